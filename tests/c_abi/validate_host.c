/*
 * Host-side validation of libLouisKV, for a build with AddressSanitizer and
 * UndefinedBehaviorSanitizer on its host code: every call below must be
 * refused with the documented status before anything is launched, the
 * workspace queries must give 0 for invalid sizes and finite sizes for large
 * valid ones, and the host-only window rule must give the documented values.
 * Device pointers are stand-ins (host buffers the library never dereferences:
 * each call fails validation first).  Prints one line per failed check;
 * exit status = number of failed checks.
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "louiskv.h"

static int failures = 0;

static void expect(const char* what, int got, int want) {
  if (got != want) {
    printf("FAIL %s: status %d (%s), expected %d; last error: %s\n", what, got, louiskv_status_str(got), want,
           louiskv_last_error());
    ++failures;
  } else if (!louiskv_last_error() || (want != LOUISKV_OK && strlen(louiskv_last_error()) == 0)) {
    printf("FAIL %s: no error text\n", what);
    ++failures;
  }
}

int main(void) {
  static char buf[1 << 16];
  void* p = buf;                 /* stand-in pointer, never dereferenced */
  int32_t* ip = (int32_t*)buf;
  float* fp = (float*)buf;
  double* dp = (double*)buf;
  uint8_t* up = (uint8_t*)buf;

  if (louiskv_abi_version() != LOUISKV_ABI_VERSION) {
    printf("FAIL abi version\n");
    ++failures;
  }
  for (int st = 0; st <= 7; ++st)
    if (!louiskv_status_str(st)) {
      printf("FAIL status string %d\n", st);
      ++failures;
    }

  /* window rule (host only) */
  int32_t ev = 0, nev = 0, nl = 0, ls = 0;
  expect("window_info valid", louiskv_window_info(160, 128, 32, &ev, &nev, &nl, &ls), LOUISKV_OK);
  if (ev != 1 || nev != 2 || nl != 97 || ls != 64) {
    printf("FAIL window_info(160, 128, 32) = %d %d %d %d\n", ev, nev, nl, ls);
    ++failures;
  }
  expect("window_info ragged", louiskv_window_info(5, 100, 32, &ev, &nev, &nl, &ls), LOUISKV_ERR_SHAPE);
  expect("window_info negative step", louiskv_window_info(-1, 128, 32, &ev, &nev, &nl, &ls), LOUISKV_ERR_SHAPE);

  /* workspace queries */
  if (louiskv_cluster_prefill_workspace_size(0, 4096, 128, 64, LOUISKV_BF16) != 0 ||
      louiskv_retrieve_workspace_size(-1, 64, 16) != 0 || louiskv_retrieve_rows_workspace_size(4, 0) != 0 ||
      louiskv_decode_step_workspace_size(8, 9, 4, 1024, 2048, 128) != 0 ||
      louiskv_decode_step_workspace_size(8, LOUISKV_BF16, 16, 1024, 2048, 128) != 0 ||
      louiskv_sparse_decode_attn_rows_workspace_size(8, 4, 128, -1, 128) != 0) {
    printf("FAIL workspace query for invalid sizes is not 0\n");
    ++failures;
  }
  if (louiskv_cluster_prefill_workspace_size(1024, 131072, 128, 4096, LOUISKV_BF16) == 0 ||
      louiskv_decode_step_workspace_size(1024, LOUISKV_BF16, 4, 8192, 8192, 128) == 0 ||
      louiskv_retrieve_delta_workspace_size(1024, 8192, 4096) == 0) {
    printf("FAIL workspace query for large valid sizes is 0\n");
    ++failures;
  }

  /* k-means prefill */
  expect("cluster_prefill NULL keys",
         louiskv_cluster_prefill(NULL, LOUISKV_BF16, 8, 4096, 128, 64, 10, ip, fp, 64, ip, ip, ip, ip, NULL, NULL,
                                 NULL, 0, 0, NULL, p, sizeof(buf), NULL), LOUISKV_ERR_NULL);
  expect("cluster_prefill dtype",
         louiskv_cluster_prefill(p, 7, 8, 4096, 128, 64, 10, ip, fp, 64, ip, ip, ip, ip, NULL, NULL, NULL, 0, 0,
                                 NULL, p, sizeof(buf), NULL), LOUISKV_ERR_DTYPE);
  expect("cluster_prefill head dim",
         louiskv_cluster_prefill(p, LOUISKV_BF16, 8, 4096, 64, 64, 10, ip, fp, 64, ip, ip, ip, ip, NULL, NULL, NULL,
                                 0, 0, NULL, p, sizeof(buf), NULL), LOUISKV_ERR_UNSUPPORTED);
  expect("cluster_prefill C > N",
         louiskv_cluster_prefill(p, LOUISKV_BF16, 8, 32, 128, 64, 10, ip, fp, 64, ip, ip, ip, ip, NULL, NULL, NULL,
                                 0, 0, NULL, p, sizeof(buf), NULL), LOUISKV_ERR_SHAPE);
  expect("cluster_prefill units_cap < C",
         louiskv_cluster_prefill(p, LOUISKV_BF16, 8, 4096, 128, 64, 10, ip, fp, 63, ip, ip, ip, ip, NULL, NULL, NULL,
                                 0, 0, NULL, p, sizeof(buf), NULL), LOUISKV_ERR_SHAPE);
  expect("cluster_prefill small workspace",
         louiskv_cluster_prefill(p, LOUISKV_BF16, 8, 4096, 128, 64, 10, ip, fp, 64, ip, ip, ip, ip, NULL, NULL, NULL,
                                 0, 0, NULL, p, 1, NULL), LOUISKV_ERR_WORKSPACE);
  expect("cluster_prefill host pool flag on host malloc memory",
         louiskv_cluster_prefill(p, LOUISKV_BF16, 8, 4096, 128, 64, 10, ip, fp, 64, ip, ip, ip, ip, p, p, p, 4096, 1,
                                 NULL, p, sizeof(buf), NULL), LOUISKV_ERR_UNSUPPORTED);

  /* boundary test */
  expect("boundary_check NULL q",
         louiskv_boundary_check(NULL, p, LOUISKV_BF16, 4, 32, 128, 0.9, LOUISKV_REF_ANCHOR, 0, dp, up, NULL),
         LOUISKV_ERR_NULL);
  expect("boundary_check mode",
         louiskv_boundary_check(p, p, LOUISKV_BF16, 4, 32, 128, 0.9, 5, 0, dp, up, NULL), LOUISKV_ERR_SHAPE);
  expect("boundary_check head dim",
         louiskv_boundary_check(p, p, LOUISKV_BF16, 4, 32, 100, 0.9, LOUISKV_REF_PREV, 0, dp, up, NULL),
         LOUISKV_ERR_UNSUPPORTED);

  /* store */
  expect("segment_output unit past units_cap",
         louiskv_segment_output(p, p, LOUISKV_BF16, 8, 128, p, p, 128, 128, 32, fp, ip, ip, 64, 64, p, p, 8192, 4096,
                                0, NULL), LOUISKV_ERR_SHAPE);
  expect("segment_output ragged window",
         louiskv_segment_output(p, p, LOUISKV_BF16, 8, 128, p, p, 100, 3, 32, fp, ip, ip, 64, 64, p, p, 8192, 4096,
                                0, NULL), LOUISKV_ERR_SHAPE);

  /* retrieval */
  expect("retrieve_rows no units",
         louiskv_retrieve_rows(p, LOUISKV_BF16, 8, 8, 4, 128, 0.088, fp, ip, ip, 64, 0, 128, up, ip, ip, ip, ip, dp,
                               p, sizeof(buf), NULL), LOUISKV_ERR_SHAPE);
  expect("retrieve_rows group size",
         louiskv_retrieve_rows(p, LOUISKV_BF16, 8, 8, 9, 128, 0.088, fp, ip, ip, 64, 64, 128, up, ip, ip, ip, ip, dp,
                               p, sizeof(buf), NULL), LOUISKV_ERR_UNSUPPORTED);
  expect("retrieve_rows small workspace",
         louiskv_retrieve_rows(p, LOUISKV_BF16, 8, 8, 4, 128, 0.088, fp, ip, ip, 1024, 1024, 2048, up, ip, ip, ip,
                               ip, dp, p, 16, NULL), LOUISKV_ERR_WORKSPACE);
  expect("retrieve_delta NULL buffers",
         louiskv_retrieve_delta(p, LOUISKV_BF16, 8, 8, 4, 128, 0.088, fp, ip, ip, 64, 64, NULL, 128, p, p, 4096, 0,
                                256, up, ip, ip, ip, NULL, NULL, ip, ip, ip, dp, p, sizeof(buf), NULL),
         LOUISKV_ERR_NULL);
  expect("retrieve_cached NULL slot_step",
         louiskv_retrieve_cached(p, LOUISKV_BF16, 8, 8, 4, 128, 0.088, fp, ip, ip, 64, 64, NULL, 128, p, p, 4096, 0,
                                 256, 1024, 5, up, ip, ip, ip, p, p, ip, NULL, ip, ip, dp, p, sizeof(buf), NULL),
         LOUISKV_ERR_NULL);
  expect("retrieve_cached cache below the budget",
         louiskv_retrieve_cached(p, LOUISKV_BF16, 8, 8, 4, 128, 0.088, fp, ip, ip, 64, 64, NULL, 128, p, p, 4096, 0,
                                 256, 128, 5, up, ip, ip, ip, p, p, ip, ip, ip, ip, dp, p, sizeof(buf), NULL),
         LOUISKV_ERR_SHAPE);
  expect("retrieve_cached cache beyond the plan's register runs",
         louiskv_retrieve_cached(p, LOUISKV_BF16, 8, 8, 4, 128, 0.088, fp, ip, ip, 64, 64, NULL, 128, p, p, 4096, 0,
                                 256, 70000, 5, up, ip, ip, ip, p, p, ip, ip, ip, ip, dp, p, sizeof(buf), NULL),
         LOUISKV_ERR_UNSUPPORTED);

  /* attention */
  expect("attn_rows group size",
         louiskv_sparse_decode_attn_rows(p, LOUISKV_BF16, 8, 8, 3, 128, 0.088f, p, p, 4096, ip, ip, 256, p, p, 128,
                                         0, 16, p, LOUISKV_F32, fp, p, sizeof(buf), NULL), LOUISKV_ERR_UNSUPPORTED);
  expect("attn_rows live rows beyond the window",
         louiskv_sparse_decode_attn_rows(p, LOUISKV_BF16, 8, 8, 4, 128, 0.088f, p, p, 4096, ip, ip, 256, p, p, 128,
                                         0, 129, p, LOUISKV_F32, fp, p, sizeof(buf), NULL), LOUISKV_ERR_SHAPE);
  expect("attn_rows small workspace",
         louiskv_sparse_decode_attn_rows(p, LOUISKV_BF16, 8, 8, 4, 128, 0.088f, p, p, 4096, ip, ip, 2048, p, p, 128,
                                         0, 16, p, LOUISKV_F32, fp, p, 8, NULL), LOUISKV_ERR_WORKSPACE);
  expect("attn_rows_noalloc partials beyond the scratch array",
         louiskv_sparse_decode_attn_rows_noalloc(p, LOUISKV_BF16, 512, 8, 4, 128, 0.088f, p, p, 4096, ip, ip,
                                                 73728, p, p, 32, 0, 0, p, LOUISKV_F32, fp, NULL),
         LOUISKV_ERR_WORKSPACE);

  /* the two-launch decode step */
  expect("decode_step NULL q",
         louiskv_decode_step(NULL, p, LOUISKV_BF16, 1, 32, 8, 128, 0.9, LOUISKV_REF_ANCHOR, 0, dp, up, p, p, p, p,
                             128, 32, fp, ip, ip, 1024, 1024, p, p, 34000, 32768, 2048, ip, ip, ip, ip, dp, p,
                             LOUISKV_F32, fp, p, sizeof(buf), NULL), LOUISKV_ERR_NULL);
  expect("decode_step group size 3",
         louiskv_decode_step(p, p, LOUISKV_BF16, 1, 24, 8, 128, 0.9, LOUISKV_REF_ANCHOR, 0, dp, up, p, p, p, p, 128,
                             32, fp, ip, ip, 1024, 1024, p, p, 34000, 32768, 2048, ip, ip, ip, ip, dp, p,
                             LOUISKV_F32, fp, p, sizeof(buf), NULL), LOUISKV_ERR_UNSUPPORTED);
  expect("decode_step ragged window",
         louiskv_decode_step(p, p, LOUISKV_BF16, 1, 32, 8, 128, 0.9, LOUISKV_REF_ANCHOR, 3, dp, up, p, p, p, p, 100,
                             32, fp, ip, ip, 1024, 1024, p, p, 34000, 32768, 2048, ip, ip, ip, ip, dp, p,
                             LOUISKV_F32, fp, p, sizeof(buf), NULL), LOUISKV_ERR_SHAPE);
  expect("decode_step units past units_cap",
         louiskv_decode_step(p, p, LOUISKV_BF16, 1, 32, 8, 128, 0.9, LOUISKV_REF_ANCHOR, 300, dp, up, p, p, p, p,
                             128, 32, fp, ip, ip, 1024, 1024, p, p, 34000, 32768, 2048, ip, ip, ip, ip, dp, p,
                             LOUISKV_F32, fp, p, sizeof(buf), NULL), LOUISKV_ERR_SHAPE);
  expect("decode_step small workspace",
         louiskv_decode_step(p, p, LOUISKV_BF16, 1, 32, 8, 128, 0.9, LOUISKV_REF_ANCHOR, 5, dp, up, p, p, p, p, 128,
                             32, fp, ip, ip, 1024, 1024, p, p, 34000, 32768, 2048, ip, ip, ip, ip, dp, p,
                             LOUISKV_F32, fp, p, 64, NULL), LOUISKV_ERR_WORKSPACE);

  /* the decode step with the LRU cache of pool rows */
  if (louiskv_decode_step_cached_workspace_size(8, LOUISKV_BF16, 4, 1024, 0, 128) != 0 ||
      louiskv_decode_step_cached_workspace_size(8, LOUISKV_BF16, 4, 1024, 2048, 128) == 0) {
    printf("FAIL decode_step_cached_workspace_size\n");
    ++failures;
  }
  expect("decode_step_cached NULL k_buf",
         louiskv_decode_step_cached(p, p, LOUISKV_BF16, 1, 32, 8, 128, 0.9, LOUISKV_REF_ANCHOR, 5, dp, up, p, p, p,
                                    p, 128, 32, fp, ip, ip, 1024, 1024, p, p, 34000, 0, 32768, 2048, 4096, NULL, p,
                                    ip, ip, ip, ip, ip, ip, ip, ip, dp, p, LOUISKV_F32, fp, p, sizeof(buf), NULL),
         LOUISKV_ERR_NULL);
  expect("decode_step_cached cache below the budget",
         louiskv_decode_step_cached(p, p, LOUISKV_BF16, 1, 32, 8, 128, 0.9, LOUISKV_REF_ANCHOR, 5, dp, up, p, p, p,
                                    p, 128, 32, fp, ip, ip, 1024, 1024, p, p, 34000, 0, 32768, 2048, 1024, p, p,
                                    ip, ip, ip, ip, ip, ip, ip, ip, dp, p, LOUISKV_F32, fp, p, sizeof(buf), NULL),
         LOUISKV_ERR_SHAPE);
  expect("decode_step_cached pool beyond the plan's bitmap",
         louiskv_decode_step_cached(p, p, LOUISKV_BF16, 1, 32, 8, 128, 0.9, LOUISKV_REF_ANCHOR, 5, dp, up, p, p, p,
                                    p, 128, 32, fp, ip, ip, 1024, 1024, p, p, 600000, 0, 32768, 2048, 4096, p, p,
                                    ip, ip, ip, ip, ip, ip, ip, ip, dp, p, LOUISKV_F32, fp, p, sizeof(buf), NULL),
         LOUISKV_ERR_UNSUPPORTED);

  printf("%d failed checks\n", failures);
  return failures;
}
