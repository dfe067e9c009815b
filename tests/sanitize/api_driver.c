/* Exercises the host side of libgdn (argument checks, packed-sequence
 * validation, workspace sizing and carving, the pointer audit) under the
 * sanitizers it is built with.  Every call here returns before its first
 * HIP call, so no GPU is needed.  Exit status 0 on success. */
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include "../../include/gdn.h"

static int fails = 0;
#define EXPECT(cond)                                              \
  do {                                                            \
    if (!(cond)) {                                                \
      fprintf(stderr, "%s:%d: expected %s\n", __FILE__, __LINE__, #cond); \
      ++fails;                                                    \
    }                                                             \
  } while (0)

static gdn_problem dense(int B, int T, int H, int dk, int dv, int dtype) {
  gdn_problem p;
  memset(&p, 0, sizeof p);
  p.B = B;
  p.T = T;
  p.H = H;
  p.dk = dk;
  p.dv = dv;
  p.dtype = (gdn_dtype)dtype;
  return p;
}

int main(void) {
  void *fake = (void *)0x10000, *odd = (void *)0x10008;
  const int dims[][2] = {{64, 64}, {128, 128}, {256, 512}, {96, 64}};
  for (int d = 0; d < 4; ++d)
    for (int T = 1; T <= 300; T += 37) {
      gdn_problem p = dense(2, T, 3, dims[d][0], dims[d][1], GDN_BF16);
      size_t f = gdn_chunk_fwd_workspace_size(&p), b = gdn_chunk_bwd_workspace_size(&p);
      size_t s = gdn_chunk_saved_size(&p), fs = gdn_chunk_fwd_save_workspace_size(&p);
      size_t bs = gdn_chunk_bwd_saved_workspace_size(&p);
      size_t blk = gdn_block_bwd_saved_workspace_size(&p, 4);
      if (d == 3) {
        EXPECT(f == 0 && b == 0 && s == 0 && fs == 0 && bs == 0 && blk == 0);
        continue;
      }
      EXPECT(f > 0 && b > f && s > 0 && fs > 0 && bs > 0 && blk > bs);
      EXPECT(gdn_chunk_fwd(&p, fake, fake, fake, fake, fake, NULL, fake, NULL, fake, f - 1,
                           NULL) == GDN_ERR_WORKSPACE);
      EXPECT(gdn_chunk_fwd(&p, NULL, fake, fake, fake, fake, NULL, fake, NULL, fake, f, NULL) ==
             GDN_ERR_NULL);
      EXPECT(gdn_chunk_fwd(&p, odd, fake, fake, fake, fake, NULL, fake, NULL, fake, f, NULL) ==
             GDN_ERR_ALIGN);
      EXPECT(gdn_chunk_bwd_saved(&p, fake, fake, fake, fake, fake, NULL, fake, s - 1, fake, fake,
                                 fake, fake, NULL, NULL, fake, bs, NULL) == GDN_ERR_SAVED);
    }
  /* packed boundaries: valid ones are sized, invalid ones rejected */
  {
    const int32_t good[] = {0, 0, 1, 65, 128, 300};
    const int32_t decreasing[] = {0, 70, 65, 300};
    const int32_t short_end[] = {0, 10, 299};
    gdn_problem p = dense(1, 300, 2, 128, 128, GDN_BF16);
    p.cu_seqlens = (const int32_t *)fake;
    p.cu_seqlens_host = good;
    p.num_seqs = 5;
    EXPECT(gdn_chunk_fwd_workspace_size(&p) > 0);
    EXPECT(gdn_block_bwd_saved_workspace_size(&p, 2) > 0);
    p.cu_seqlens_host = decreasing;
    p.num_seqs = 3;
    EXPECT(gdn_chunk_fwd_workspace_size(&p) == 0);
    EXPECT(gdn_chunk_fwd(&p, fake, fake, fake, fake, fake, NULL, fake, NULL, fake, 1 << 30,
                         NULL) == GDN_ERR_CU_SEQLENS);
    p.cu_seqlens_host = short_end;
    p.num_seqs = 2;
    EXPECT(gdn_chunk_fwd_workspace_size(&p) == 0);
    p.cu_seqlens_host = NULL;
    EXPECT(gdn_chunk_fwd(&p, fake, fake, fake, fake, fake, NULL, fake, NULL, fake, 1 << 30,
                         NULL) == GDN_ERR_CU_SEQLENS);
    gdn_problem q = dense(2, 300, 2, 128, 128, GDN_BF16);  /* packed needs B == 1 */
    q.cu_seqlens = (const int32_t *)fake;
    q.cu_seqlens_host = good;
    q.num_seqs = 5;
    EXPECT(gdn_chunk_fwd_workspace_size(&q) == 0);
  }
  /* shapes and dtypes outside the supported set */
  {
    gdn_problem p = dense(1, 64, 1, 256, 256, GDN_F32);
    EXPECT(gdn_chunk_fwd_workspace_size(&p) == 0);
    p = dense(1, 64, 1, 256, 512, GDN_F32);
    EXPECT(gdn_chunk_fwd_workspace_size(&p) > 0);
    p = dense(0, 64, 1, 64, 64, GDN_BF16);
    EXPECT(gdn_chunk_fwd(&p, fake, fake, fake, fake, fake, NULL, fake, NULL, fake, 1, NULL) ==
           GDN_ERR_SHAPE);
    p = dense(1 << 20, 1 << 12, 1, 64, 64, GDN_BF16);
    EXPECT(gdn_chunk_fwd_workspace_size(&p) == 0);
    EXPECT(gdn_chunk_fwd(NULL, fake, fake, fake, fake, fake, NULL, fake, NULL, fake, 1, NULL) ==
           GDN_ERR_NULL);
  }
  /* the no-allocation forward refuses what its array cannot hold */
  {
    gdn_problem p = dense(8, 4096, 6, 256, 512, GDN_BF16);
    EXPECT(gdn_chunk_fwd_noalloc(&p, fake, fake, fake, fake, fake, NULL, fake, NULL, NULL) ==
           GDN_ERR_WORKSPACE);
  }
  /* fused block: prologue checks */
  {
    gdn_problem p = dense(2, 100, 3, 64, 64, GDN_BF16);
    gdn_block_prologue pro = {4, 1e-6f, fake, fake, fake, fake, fake, fake};
    size_t f = gdn_chunk_fwd_workspace_size(&p);
    EXPECT(gdn_block_fwd(&p, &pro, fake, fake, NULL, fake, NULL, NULL, NULL, NULL, fake, f - 1,
                         NULL) == GDN_ERR_WORKSPACE);
    pro.width = 9;
    EXPECT(gdn_block_fwd(&p, &pro, fake, fake, NULL, fake, NULL, NULL, NULL, NULL, fake, f,
                         NULL) == GDN_ERR_VALUE);
    pro.width = 2;
    pro.xk = NULL;
    EXPECT(gdn_block_fwd(&p, &pro, fake, fake, NULL, fake, NULL, NULL, NULL, NULL, fake, f,
                         NULL) == GDN_ERR_NULL);
  }
  /* the pointer audit over every sequence and single missing field */
  for (int seq = 0; seq < 8; ++seq) {
    int n = 0;
    while (gdn_debug_audit_field(n)) ++n;
    const uint64_t all = n == 64 ? ~0ull : (1ull << n) - 1;
    EXPECT(gdn_debug_audit(seq, all) == -1);
    for (int i = 0; i < n; ++i) {
      const int r = gdn_debug_audit(seq, all & ~(1ull << i));
      EXPECT(r == -1 || r == i);
    }
  }
  EXPECT(gdn_debug_audit(-1, 0) == -2);
  for (int c = 0; c <= 9; ++c) EXPECT(gdn_status_string((gdn_status)c) != NULL);
  printf(fails ? "api driver: %d FAILED\n" : "api driver: ok\n", fails);
  return fails ? 1 : 0;
}
