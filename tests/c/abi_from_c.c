/* A plain C99 caller of the SSBA C ABI: includes every public header and
 * calls the entry points that need no device (version, status strings,
 * workspace sizes, argument rejection).  Exits 0 when every check holds,
 * otherwise prints the failing check and exits 1. */
#include <stdio.h>
#include <string.h>

#include "ssba.h"
#include "ssba_haar.h"
#include "ssba_probe.h"

#define CHECK(cond)                                              \
  do {                                                           \
    if (!(cond)) {                                               \
      fprintf(stderr, "check failed: %s (line %d)\n", #cond, __LINE__); \
      return 1;                                                  \
    }                                                            \
  } while (0)

int main(void) {
  ssba_desc d;
  size_t index_bytes = 0, scratch_bytes = 0;
  memset(&d, 0, sizeof d);
  d.batch = 1;
  d.heads = 16;
  d.head_dim = 64;
  d.grid_h = 64;
  d.grid_w = 64;
  d.tile = 8;
  d.shift_y = 4;
  d.shift_x = 4;
  d.gate = SSBA_GATE_WINDOW;
  d.win_h = 2;
  d.win_w = 2;
  d.dtype = SSBA_DT_BF16;

  CHECK(ssba_abi_version() == SSBA_ABI_VERSION);
  CHECK(ssba_status_str(SSBA_OK) != NULL && ssba_status_str((ssba_status)99) != NULL);

  /* window gate: only the per-row status flags */
  CHECK(ssba_workspace_size(&d, &index_bytes, &scratch_bytes) == SSBA_OK);
  CHECK(index_bytes == (size_t)4 * 16 * 64 * 65);
  CHECK(scratch_bytes == (size_t)4 * 16 * 64);

  /* top-k gate: pooled sums in fp64 plus the flags */
  d.gate = SSBA_GATE_TOPK;
  d.keep = 10;
  CHECK(ssba_workspace_size(&d, NULL, &scratch_bytes) == SSBA_OK);
  CHECK(scratch_bytes == (size_t)16 * 16 * 64 * 64 + (size_t)4 * 16 * 64);

  /* rejected before any launch */
  d.keep = 0;
  CHECK(ssba_workspace_size(&d, &index_bytes, &scratch_bytes) == SSBA_ERR_ARG);
  d.keep = 10;
  d.grid_w = 60;
  CHECK(ssba_workspace_size(&d, &index_bytes, &scratch_bytes) == SSBA_ERR_SHAPE);
  d.grid_w = 64;
  d.head_dim = 96;
  CHECK(ssba_workspace_size(&d, &index_bytes, &scratch_bytes) == SSBA_ERR_UNSUPPORTED);
  d.head_dim = 64;
  CHECK(ssba_build_index(&d, NULL, NULL, NULL, NULL, NULL) == SSBA_ERR_ARG);
  CHECK(ssba_forward(NULL, NULL, NULL, NULL, NULL, NULL, NULL) == SSBA_ERR_ARG);
  CHECK(ssba_forward_kernel(&d, 0) != NULL);

  /* short workspaces are rejected before any launch (the pointers are never
   * dereferenced: the size check precedes every launch) */
  {
    void* fake = (void*)(uintptr_t)0x100000;
    size_t ib = 0, sb = 0;
    CHECK(ssba_workspace_size(&d, &ib, &sb) == SSBA_OK);
    CHECK(ssba_build_index_ex(&d, fake, fake, (int32_t*)fake, ib - 1, fake, sb, NULL) == SSBA_ERR_WORKSPACE);
    CHECK(ssba_build_index_ex(&d, fake, fake, (int32_t*)fake, ib, fake, sb - 1, NULL) == SSBA_ERR_WORKSPACE);
    CHECK(ssba_forward_ex(&d, fake, fake, fake, (const int32_t*)fake, ib - 1, fake, NULL) == SSBA_ERR_WORKSPACE);
    CHECK(ssba_forward_topk_ex(&d, fake, fake, fake, (int32_t*)fake, ib, fake, sb - 1, fake, NULL) ==
          SSBA_ERR_WORKSPACE);
    CHECK(ssba_forward_topk_ex(&d, NULL, fake, fake, (int32_t*)fake, ib, fake, sb, fake, NULL) == SSBA_ERR_ARG);
    /* the fused call's two launches, one at a time */
    CHECK(ssba_pool_keys_ex(&d, fake, fake, sb - 1, NULL) == SSBA_ERR_WORKSPACE);
    CHECK(ssba_pool_keys_ex(&d, NULL, fake, sb, NULL) == SSBA_ERR_ARG);
    CHECK(ssba_forward_gated_ex(&d, fake, fake, fake, (int32_t*)fake, ib - 1, fake, sb, fake, NULL) ==
          SSBA_ERR_WORKSPACE);
    CHECK(ssba_forward_gated_ex(&d, fake, fake, NULL, (int32_t*)fake, ib, fake, sb, fake, NULL) == SSBA_ERR_ARG);
    d.tile = 16;
    CHECK(ssba_pool_keys_ex(&d, fake, fake, (size_t)1 << 30, NULL) == SSBA_ERR_UNSUPPORTED);
    CHECK(ssba_rope_pool_keys_ex(&d, fake, fake, fake, fake, 0.f, fake, (size_t)1 << 30, NULL) ==
          SSBA_ERR_UNSUPPORTED);
    d.tile = 8;
    /* the rotary forms */
    CHECK(ssba_rope_pool_keys_ex(&d, fake, fake, fake, fake, 0.f, fake, sb - 1, NULL) == SSBA_ERR_WORKSPACE);
    CHECK(ssba_rope_pool_keys_ex(&d, fake, fake, NULL, fake, 0.f, fake, sb, NULL) == SSBA_ERR_ARG);
    CHECK(ssba_forward_topk_rope_ex(&d, fake, fake, fake, fake, fake, 0.f, (int32_t*)fake, ib - 1, fake, sb, fake,
                                    NULL) == SSBA_ERR_WORKSPACE);
    CHECK(ssba_forward_topk_rope_ex(&d, fake, fake, fake, fake, fake, 1.0f / 0.0f, (int32_t*)fake, ib, fake, sb,
                                    fake, NULL) == SSBA_ERR_ARG);
  }
  CHECK(ssba_forward_kernel(&d, 7) == NULL);

  /* the Haar pair and the probe reject bad arguments the same way */
  {
    ssba_haar_desc h;
    memset(&h, 0, sizeof h);
    CHECK(ssba_haar_kernel_name(&h, 0) == NULL);
  }
  CHECK(ssba_probe_mfma(0, 10, NULL, NULL) == SSBA_ERR_ARG);

  printf("ok\n");
  return 0;
}
