/* C99 client of the VisionPulse C ABI: host-side calls only (no device is
 * needed): status strings, shape validation, workspace sizing, launch plans
 * and the host mirror of the Eq. (7) budget rule. Exits non-zero on the first
 * failed check, printing it. */
#include <stdio.h>
#include <string.h>

#include "visionpulse.h"

static int failures = 0;
#define CHECK(cond)                                                   \
  do {                                                                \
    if (!(cond)) {                                                    \
      fprintf(stderr, "%s:%d: check failed: %s\n", __FILE__, __LINE__, #cond); \
      ++failures;                                                     \
    }                                                                 \
  } while (0)

static vp_shape shape_7b(void) {
  vp_shape s;
  memset(&s, 0, sizeof(s));
  s.batch = 1;
  s.n_q_heads = 28;
  s.n_kv_heads = 4;
  s.head_dim = 128;
  s.dtype = VP_BF16;
  s.max_seq_len = 3358;
  s.max_vis = 1296;
  s.max_segs = 1;
  s.k_cap = 64;
  s.kv_stride_h = 3358 * 128;
  s.kv_stride_b = 4 * s.kv_stride_h;
  s.kv_stride_s = 128;
  return s;
}

int main(void) {
  CHECK(strcmp(vp_status_string(VP_OK), "VP_OK") == 0);
  CHECK(strcmp(vp_status_string(VP_ERR_WORKSPACE), "VP_ERR_WORKSPACE") == 0);

  /* workspace sizing: valid shapes */
  vp_shape s = shape_7b();
  size_t bytes = 0;
  CHECK(vp_workspace_size(&s, &bytes) == VP_OK);
  CHECK(bytes > 0 && bytes % 256 == 0);
  size_t one = bytes;
  s.n_queries = 2; /* two queries per sequence: 14 query rows per KV head */
  CHECK(vp_workspace_size(&s, &bytes) == VP_OK && bytes > one);
  s = shape_7b();
  s.scope = VP_SCOPE_KV_GROUP;
  CHECK(vp_workspace_size(&s, &bytes) == VP_OK);

  /* validation: each error names itself in vp_last_error */
  s = shape_7b();
  s.n_q_heads = 30;
  CHECK(vp_workspace_size(&s, &bytes) == VP_ERR_SHAPE);
  CHECK(strlen(vp_last_error()) > 0);
  s = shape_7b();
  s.head_dim = 96;
  CHECK(vp_workspace_size(&s, &bytes) == VP_ERR_UNSUPPORTED);
  s = shape_7b();
  s.n_queries = 3; /* 21 query rows per KV head > 16 */
  CHECK(vp_workspace_size(&s, &bytes) == VP_ERR_UNSUPPORTED);
  s = shape_7b();
  s.dtype = 9;
  CHECK(vp_workspace_size(&s, &bytes) == VP_ERR_DTYPE);
  s = shape_7b();
  CHECK(vp_workspace_size(&s, NULL) == VP_ERR_NULL);
  CHECK(vp_workspace_size(NULL, &bytes) == VP_ERR_NULL);

  /* launch plan of the 7B batch-1 step: one context launch, chunked selection */
  vp_params p;
  memset(&p, 0, sizeof(p));
  p.tau_mass = 0.1f;
  p.tau_score = 1.0f;
  p.r_lo_bp = 100;
  p.r_hi_bp = 500;
  p.clamp = 1;
  int32_t flags = -1;
  s = shape_7b();
  CHECK(vp_step_plan(&s, &p, &flags) == VP_OK);
  CHECK((flags & VP_PLAN_ONE_CONTEXT_LAUNCH) != 0);

  /* Eq. (7) with the Sec. 5.2 clamp: 1296 visual tokens, clamp [13, 64] */
  CHECK(vp_budget_host(0.0, 1296, &p) == 13);
  CHECK(vp_budget_host(1.0, 1296, &p) == 64);
  CHECK(vp_budget_host(0.03, 1296, &p) == 39);   /* ceil(38.88) */
  CHECK(vp_budget_host(0.5, 0, &p) == 0);
  p.clamp = 0;
  CHECK(vp_budget_host(0.25, 1296, &p) == 324);  /* exact product: no rounding up */
  CHECK(vp_budget_host(1.0, 1296, &p) == 1296);
  p.tau_mass = 0.0f;
  CHECK(vp_budget_host(0.5, 100, &p) == -1);     /* invalid parameters */

  /* every call rejects bad arguments before touching the device */
  p.clamp = 1;
  p.tau_mass = 0.1f;
  vp_layout lay;
  memset(&lay, 0, sizeof(lay));
  int32_t dummy[4] = {0, 0, 0, 0};
  lay.seq_len = dummy;
  lay.vis_seg_off = dummy;
  lay.vis_seg = dummy;
  s = shape_7b();
  CHECK(vp_workspace_size(&s, &bytes) == VP_OK);
  CHECK(vp_decode_step(&s, &lay, &p, NULL, dummy, dummy, NULL, NULL, NULL, NULL, NULL, NULL, NULL, bytes, NULL,
                       NULL, 0) == VP_ERR_NULL);
  CHECK(vp_visual_mass(&s, NULL, &p, dummy, dummy, NULL, NULL, NULL, NULL, NULL, bytes, NULL) == VP_ERR_NULL);
  CHECK(vp_budget(&s, &lay, &p, NULL, NULL, NULL) == VP_ERR_NULL);
  CHECK(vp_select_topk(&s, &lay, NULL, NULL, NULL, NULL) == VP_ERR_NULL);
  CHECK(vp_budget_top_p(&s, &lay, (const float*)dummy, 2.0f, dummy, NULL) == VP_ERR_RANGE);
  CHECK(vp_validate_layout(&s, NULL, NULL) == VP_ERR_NULL);
  s.block_size = 32; /* paged caches need a block table */
  CHECK(vp_validate_layout(&s, &lay, NULL) == VP_ERR_NULL);
  s = shape_7b();
  p.tau_mass = -1.0f;
  CHECK(vp_sparse_decode_attn(&s, &lay, &p, dummy, dummy, dummy, dummy, dummy, dummy, 0, dummy, bytes, NULL) ==
        VP_ERR_RANGE);
  p.tau_mass = 0.1f;
  CHECK(vp_sparse_decode_attn(&s, &lay, &p, dummy, dummy, dummy, dummy, dummy, dummy, 0, dummy, 16, NULL) ==
        VP_ERR_WORKSPACE);
  CHECK(strlen(vp_last_error()) > 0);

  if (failures) {
    fprintf(stderr, "%d check(s) failed\n", failures);
    return 1;
  }
  printf("C ABI smoke: all checks passed (sizeof vp_shape %zu, vp_layout %zu, vp_params %zu)\n",
         sizeof(vp_shape), sizeof(vp_layout), sizeof(vp_params));
  return 0;
}
