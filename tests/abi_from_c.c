/* Compiled as plain C99 against include/massive.h by tests/test_abi_c.py:
 * prints the byte offset and size of every field of the two ABI structs (the
 * Python binding's ctypes layouts are compared with them), then, linked
 * against libmassive.so, checks an argument error path that needs no GPU. */
#include <stddef.h>
#include <stdio.h>
#include <string.h>

#include "massive.h"

#define F(T, f) printf(#T " " #f " %zu %zu\n", offsetof(T, f), sizeof(((T*)0)->f))

int main(int argc, char** argv) {
  (void)argv;
  F(massive_init_args, L);
  F(massive_init_args, H);
  F(massive_init_args, indptr);
  F(massive_init_args, indices);
  F(massive_init_args, halo_gid);
  F(massive_init_args, halo_degree);
  F(massive_init_args, local_feat);
  F(massive_init_args, halo_store);
  F(massive_init_args, row_bytes);
  F(massive_init_args, K);
  F(massive_init_args, fanout);
  F(massive_init_args, buffer_pct);
  F(massive_init_args, gamma);
  F(massive_init_args, delta);
  F(massive_init_args, seed);
  F(massive_init_args, stream);
  F(massive_init_args, score_layout);
  F(massive_init_args, n_global);
  F(massive_init_args, link_mode);
  F(massive_init_args, link_threads);
  printf("massive_init_args sizeof %zu 0\n", sizeof(massive_init_args));
  F(massive_batch, nodes);
  F(massive_batch, mask);
  F(massive_batch, feat);
  F(massive_batch, nodes_cap);
  F(massive_batch, indptr);
  F(massive_batch, indices);
  F(massive_batch, indptr_cap);
  F(massive_batch, indices_cap);
  F(massive_batch, n);
  F(massive_batch, e);
  F(massive_batch, local);
  F(massive_batch, hits);
  F(massive_batch, misses);
  F(massive_batch, host_rows);
  printf("massive_batch sizeof %zu 0\n", sizeof(massive_batch));
  if (argc > 1) {
    /* error paths that return before any device call */
    massive_ctx* ctx = (massive_ctx*)1;
    int rc = massive_init(NULL, &ctx);
    printf("err init_null_args %d %d\n", rc, ctx == NULL);
    const char* msg = massive_last_error(NULL);
    printf("err last_error_set %d\n", msg != NULL && strlen(msg) > 0);
    printf("err sample_null_ctx %d\n", massive_sample(NULL, NULL, 0, NULL));
    printf("err destroy_null_ctx %d\n", massive_destroy(NULL));
  }
  return 0;
}
