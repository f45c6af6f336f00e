/* A plain C99 client of libdsattn.so: only the declarations of include/dsattn.h, linked
 * against the library, no GPU needed.  It prints lines the Python test compares with the
 * oracle:
 *   lambda <recall> <N> <value>
 *   order <T> <Y> <X> <bt> <by> <bx> <perm...>
 *   status <case> <return code> <message>
 *   version <string>
 */
#include <stdio.h>
#include <string.h>

#include "dsattn.h"

static void print_status(const char* name, int rc) {
  printf("status %s %d %s\n", name, rc, dsattn_last_error());
}

int main(void) {
  const float recalls[] = {0.5f, 0.9f, 0.95f, 0.99f, 1.0f};
  const int ns[] = {2048, 75600};
  for (int i = 0; i < 5; ++i)
    for (int j = 0; j < 2; ++j)
      printf("lambda %.9g %d %.9g\n", (double)recalls[i], ns[j],
             (double)dsattn_lambda_from_recall(recalls[i], ns[j]));

  int32_t perm[3 * 5 * 7];
  const int rc = dsattn_block_order(3, 5, 7, 2, 2, 3, perm);
  if (rc != DSATTN_OK) {
    print_status("block_order", rc);
    return 1;
  }
  printf("order 3 5 7 2 2 3");
  for (int i = 0; i < 3 * 5 * 7; ++i) printf(" %d", perm[i]);
  printf("\n");

  print_status("null_args", dsattn_attn_fwd_ex(NULL));

  dsattn_args a;
  memset(&a, 0, sizeof a);
  a.rule = DSATTN_RULE_DYNSPARSE_LAMBDA;
  a.param = -6.0f;
  a.B = 1;
  a.H = 2;
  a.N = 256;
  a.d = 128;
  a.scale = 0.088f;
  a.tile_q = 128;
  a.tile_k = 48;
  print_status("bad_tile", dsattn_attn_fwd_ex(&a));
  a.tile_k = 64;
  a.d = 64;
  print_status("bad_head_dim", dsattn_attn_fwd_ex(&a));
  a.d = 128;
  print_status("null_pointers", dsattn_attn_fwd_ex(&a));
  a.N = 0;
  print_status("empty", dsattn_attn_fwd_ex(&a));
  a.N = 256;
  a.rule = DSATTN_RULE_BLASST;
  a.param = 2.0f;
  print_status("bad_tau", dsattn_attn_fwd_ex(&a));
  print_status("bad_key_mean_d", dsattn_key_mean(NULL, NULL, 1, 16, 96, NULL));
  print_status("quantize_empty", dsattn_quantize_mxfp8(NULL, NULL, NULL, 0, 128, NULL));
  printf("version %s\n", dsattn_version());
  return 0;
}
