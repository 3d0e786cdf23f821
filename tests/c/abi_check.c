/* A plain C consumer of the library's C ABI: it includes kamera.h, links
 * libkamera.so and checks, with no GPU and no device memory touched, that
 * the struct layouts the header gives a C compiler match the library's, that
 * host-side validation rejects bad calls before any HIP call, and that the
 * page-table check works on a host copy.  Prints "ok" and exits 0 on success. */
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include "kamera.h"

static int failures = 0;

#define CHECK(cond)                                                        \
  do {                                                                     \
    if (!(cond)) {                                                         \
      fprintf(stderr, "FAILED %s:%d: %s (%s)\n", __FILE__, __LINE__, #cond, \
              kamera_last_error());                                        \
      ++failures;                                                          \
    }                                                                      \
  } while (0)

/* a device address that is never dereferenced: validation only */
#define FAKE ((void*)(uintptr_t)0x100000000000ull)

static void fill_rehydrate(kamera_rehydrate_args* a) {
  memset(a, 0, sizeof(*a));
  a->n_chunks = 2;
  a->n_layers = 3;
  a->n_heads = 4;
  a->head_dim = 128;
  a->n_tokens = 100;
  a->rope.theta = 1e6;
  a->rope.rope_dim = 128;
  a->rope.pairing = KAMERA_PAIR_NEOX;
  a->rope.n_sections = 1;
  a->pos_mode = KAMERA_POS_LINEAR;
  a->chunk_pos = (const int32_t*)FAKE;
  a->n_planes = 1;
  kamera_plane* p = &a->plane[0];
  const int64_t in_s[4] = {3LL * 100 * 4 * 128, 100LL * 4 * 128, 4 * 128, 128};
  p->in = (const char*)FAKE + (1ull << 32);
  memcpy(p->in_stride, in_s, sizeof(in_s));
  p->out = (char*)FAKE + (2ull << 32);
  memcpy(p->out_stride, in_s, sizeof(in_s));
  p->rotate = 1;
  p->patch_dim = 128;
}

int main(void) {
  CHECK(kamera_abi_version() == KAMERA_ABI_VERSION);
  CHECK(kamera_struct_size(0) == (int64_t)sizeof(kamera_rehydrate_args));
  CHECK(kamera_struct_size(1) == (int64_t)sizeof(kamera_shift_args));
  CHECK(kamera_struct_size(2) == (int64_t)sizeof(kamera_scatter_args));
  CHECK(kamera_struct_size(3) == (int64_t)sizeof(kamera_plane));
  CHECK(kamera_struct_size(4) == (int64_t)sizeof(kamera_rope));
  CHECK(kamera_struct_size(5) == (int64_t)sizeof(kamera_form_args));

  /* NULL argument structs */
  CHECK(kamera_rehydrate(NULL, NULL) == KAMERA_ERR_NULL);
  CHECK(strlen(kamera_last_error()) > 0);
  CHECK(kamera_shift(NULL, NULL) == KAMERA_ERR_NULL);
  CHECK(kamera_scatter_paged(NULL, NULL) == KAMERA_ERR_NULL);
  CHECK(kamera_gather_paged(NULL, NULL) == KAMERA_ERR_NULL);
  CHECK(kamera_form_patch(NULL, NULL) == KAMERA_ERR_NULL);

  /* a well-formed rehydrate passes validation; each planted fault is caught */
  kamera_rehydrate_args a;
  fill_rehydrate(&a);
  CHECK(kamera_validate(0, &a) == KAMERA_OK);
  CHECK(strlen(kamera_last_error()) == 0);
  fill_rehydrate(&a);
  a.rope.rope_dim = 127;
  CHECK(kamera_validate(0, &a) == KAMERA_ERR_SHAPE);
  fill_rehydrate(&a);
  a.plane[0].in = (const char*)a.plane[0].in + 2;
  CHECK(kamera_validate(0, &a) == KAMERA_ERR_ALIGN);
  fill_rehydrate(&a);
  a.plane[0].m = KAMERA_MAX_RANK + 1;
  CHECK(kamera_validate(0, &a) == KAMERA_ERR_RANGE);
  fill_rehydrate(&a);
  a.plane[0].out = (char*)a.plane[0].in + 256; /* overlaps its input, not exactly in place */
  CHECK(kamera_validate(0, &a) == KAMERA_ERR_ALIAS);
  fill_rehydrate(&a);
  a.plane[0].out = (void*)a.plane[0].in; /* exactly in place */
  CHECK(kamera_validate(0, &a) == KAMERA_OK);
  /* a rejected launch returns the same code as its validation */
  fill_rehydrate(&a);
  a.rope.n_sections = 2;
  CHECK(kamera_rehydrate(&a, NULL) == KAMERA_ERR_SHAPE);

  /* kernel plan: AUTO keeps this small grid on the per-head kernel; the
   * row-group kernel when requested; an unknown choice is rejected */
  fill_rehydrate(&a);
  CHECK(kamera_rehydrate_plan(&a) == KAMERA_PLAN_PER_HEAD);
  a.kernel = KAMERA_KERNEL_ROW_GROUP;   /* 4 heads: one 4-head group per row */
  CHECK(kamera_rehydrate_plan(&a) == KAMERA_PLAN_ROW_GROUP4);
  a.kernel = KAMERA_KERNEL_ROW_GROUP4;
  CHECK(kamera_rehydrate_plan(&a) == KAMERA_PLAN_ROW_GROUP4);
  a.kernel = 9;
  CHECK(kamera_rehydrate_plan(&a) == KAMERA_ERR_SHAPE);
  fill_rehydrate(&a);
  a.n_tokens = 0;
  CHECK(kamera_rehydrate_plan(&a) == KAMERA_PLAN_NONE);
  CHECK(kamera_rehydrate_schedule(&a) == 0);

  /* row-group schedule: none for the per-head kernel; a small grid runs
   * persistent under AUTO; blocks on request, but not with a cap */
  fill_rehydrate(&a);
  CHECK(kamera_rehydrate_schedule(&a) == 0);
  a.kernel = KAMERA_KERNEL_ROW_GROUP4;
  CHECK(kamera_rehydrate_schedule(&a) == KAMERA_SCHEDULE_PERSISTENT);
  a.schedule = KAMERA_SCHEDULE_BLOCKS;
  CHECK(kamera_rehydrate_schedule(&a) == KAMERA_SCHEDULE_BLOCKS);
  a.max_workgroups = 4;
  CHECK(kamera_rehydrate_schedule(&a) == KAMERA_ERR_SHAPE);
  a.schedule = 5;
  a.max_workgroups = 0;
  CHECK(kamera_rehydrate_schedule(&a) == KAMERA_ERR_SHAPE);

  /* page-table check on a host copy: 2 chunks x 3 pages of 16 tokens */
  int32_t pt[6] = {5, 1, 2, 0, 4, 3};
  CHECK(kamera_check_page_table(pt, 2, 3, 40, 16, 6) == KAMERA_OK);
  pt[4] = 1;
  CHECK(kamera_check_page_table(pt, 2, 3, 40, 16, 6) == KAMERA_ERR_ALIAS);
  pt[4] = 6;
  CHECK(kamera_check_page_table(pt, 2, 3, 40, 16, 6) == KAMERA_ERR_RANGE);

  /* patch forming: dim must be a multiple of 4 */
  kamera_form_args f;
  memset(&f, 0, sizeof(f));
  f.n_chunks = f.n_layers = f.n_heads = 1;
  f.n_tokens = 10;
  f.dim = 30;
  f.m = 2;
  CHECK(kamera_validate(4, &f) == KAMERA_ERR_UNSUPPORTED);
  CHECK(kamera_validate(7, &f) != KAMERA_OK);

  if (failures) return 1;
  printf("ok\n");
  return 0;
}
