/* Runs attention through the C ABI from plain C: device buffers come from hipMalloc, the
 * call uses the default stream, results are copied back and written to files.
 *
 *   dsattn_gpu_client DIR B H N LAMBDA TILE_Q
 *
 * DIR holds q.bin, k.bin and v.bin (bf16 [B][H][N][128], little endian).  Written to DIR:
 * o.bin (bf16), mask.bin (uint8 [B*H][ceil(N/TILE_Q)][ceil(N/64)]), lse.bin (float32
 * [B*H][N]), stats.bin (uint64 [B*H][4]) from dsattn_attn_fwd_ex with the DynSparse rule
 * at LAMBDA, and o_named.bin from dynsparse_attn_fwd_lambda with the same arguments. */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <hip/hip_runtime_api.h>

#include "dsattn.h"

static int check_hip(hipError_t e, const char* what) {
  if (e != hipSuccess) {
    fprintf(stderr, "%s: %s\n", what, hipGetErrorString(e));
    return 1;
  }
  return 0;
}

static void* read_file(const char* dir, const char* name, size_t bytes) {
  char path[1024];
  snprintf(path, sizeof path, "%s/%s", dir, name);
  FILE* f = fopen(path, "rb");
  if (f == NULL) return NULL;
  void* p = malloc(bytes);
  size_t got = p != NULL ? fread(p, 1, bytes, f) : 0;
  fclose(f);
  if (got != bytes) {
    free(p);
    return NULL;
  }
  return p;
}

static int write_file(const char* dir, const char* name, const void* p, size_t bytes) {
  char path[1024];
  snprintf(path, sizeof path, "%s/%s", dir, name);
  FILE* f = fopen(path, "wb");
  if (f == NULL) return 1;
  size_t put = fwrite(p, 1, bytes, f);
  fclose(f);
  return put != bytes;
}

int main(int argc, char** argv) {
  if (argc != 7) {
    fprintf(stderr, "usage: %s DIR B H N LAMBDA TILE_Q\n", argv[0]);
    return 2;
  }
  const char* dir = argv[1];
  const int B = atoi(argv[2]), H = atoi(argv[3]), N = atoi(argv[4]);
  const float lambda = (float)atof(argv[5]);
  const int tile_q = atoi(argv[6]), tile_k = 64, d = 128;
  const size_t elems = (size_t)B * H * N * d;
  const size_t n_mask = (size_t)B * H * ((N + tile_q - 1) / tile_q) * ((N + tile_k - 1) / tile_k);
  const size_t n_lse = (size_t)B * H * N, n_stats = (size_t)B * H * 4;

  void* hq = read_file(dir, "q.bin", elems * 2);
  void* hk = read_file(dir, "k.bin", elems * 2);
  void* hv = read_file(dir, "v.bin", elems * 2);
  if (hq == NULL || hk == NULL || hv == NULL) {
    fprintf(stderr, "cannot read q/k/v from %s\n", dir);
    return 1;
  }
  void *dq, *dk, *dv, *dout, *dnamed, *dmask, *dlse, *dstats;
  if (check_hip(hipMalloc(&dq, elems * 2), "hipMalloc") ||
      check_hip(hipMalloc(&dk, elems * 2), "hipMalloc") ||
      check_hip(hipMalloc(&dv, elems * 2), "hipMalloc") ||
      check_hip(hipMalloc(&dout, elems * 2), "hipMalloc") ||
      check_hip(hipMalloc(&dnamed, elems * 2), "hipMalloc") ||
      check_hip(hipMalloc(&dmask, n_mask), "hipMalloc") ||
      check_hip(hipMalloc(&dlse, n_lse * 4), "hipMalloc") ||
      check_hip(hipMalloc(&dstats, n_stats * 8), "hipMalloc"))
    return 1;
  if (check_hip(hipMemcpy(dq, hq, elems * 2, hipMemcpyHostToDevice), "copy q") ||
      check_hip(hipMemcpy(dk, hk, elems * 2, hipMemcpyHostToDevice), "copy k") ||
      check_hip(hipMemcpy(dv, hv, elems * 2, hipMemcpyHostToDevice), "copy v"))
    return 1;

  const float scale = 0.08838834764831845f; /* 1 / sqrt(128) */
  dsattn_args a;
  memset(&a, 0, sizeof a);
  a.rule = DSATTN_RULE_DYNSPARSE_LAMBDA;
  a.param = lambda;
  a.q = dq;
  a.k = dk;
  a.v = dv;
  a.o = dout;
  a.B = B;
  a.H = H;
  a.N = N;
  a.d = d;
  a.scale = scale;
  a.tile_q = tile_q;
  a.tile_k = tile_k;
  a.stream = NULL;
  a.stats_out = (uint64_t*)dstats;
  a.mask_out = (uint8_t*)dmask;
  a.lse_out = (float*)dlse;
  a.key_order = DSATTN_ORDER_ASCENDING;
  a.qk_format = DSATTN_QK_BF16;
  int rc = dsattn_attn_fwd_ex(&a);
  if (rc != DSATTN_OK) {
    fprintf(stderr, "dsattn_attn_fwd_ex: %d %s\n", rc, dsattn_last_error());
    return 1;
  }
  rc = dynsparse_attn_fwd_lambda(dq, dk, dv, dnamed, B, H, N, d, scale, lambda, tile_q, tile_k,
                                 NULL, NULL);
  if (rc != DSATTN_OK) {
    fprintf(stderr, "dynsparse_attn_fwd_lambda: %d %s\n", rc, dsattn_last_error());
    return 1;
  }
  if (check_hip(hipDeviceSynchronize(), "synchronize")) return 1;

  void* ho = malloc(elems * 2);
  void* hn = malloc(elems * 2);
  void* hm = malloc(n_mask);
  void* hl = malloc(n_lse * 4);
  void* hs = malloc(n_stats * 8);
  if (ho == NULL || hn == NULL || hm == NULL || hl == NULL || hs == NULL) return 1;
  if (check_hip(hipMemcpy(ho, dout, elems * 2, hipMemcpyDeviceToHost), "copy o") ||
      check_hip(hipMemcpy(hn, dnamed, elems * 2, hipMemcpyDeviceToHost), "copy o_named") ||
      check_hip(hipMemcpy(hm, dmask, n_mask, hipMemcpyDeviceToHost), "copy mask") ||
      check_hip(hipMemcpy(hl, dlse, n_lse * 4, hipMemcpyDeviceToHost), "copy lse") ||
      check_hip(hipMemcpy(hs, dstats, n_stats * 8, hipMemcpyDeviceToHost), "copy stats"))
    return 1;
  if (write_file(dir, "o.bin", ho, elems * 2) || write_file(dir, "o_named.bin", hn, elems * 2) ||
      write_file(dir, "mask.bin", hm, n_mask) || write_file(dir, "lse.bin", hl, n_lse * 4) ||
      write_file(dir, "stats.bin", hs, n_stats * 8)) {
    fprintf(stderr, "cannot write results to %s\n", dir);
    return 1;
  }
  hipFree(dq); hipFree(dk); hipFree(dv); hipFree(dout); hipFree(dnamed);
  hipFree(dmask); hipFree(dlse); hipFree(dstats);
  free(hq); free(hk); free(hv); free(ho); free(hn); free(hm); free(hl); free(hs);
  printf("ok\n");
  return 0;
}
