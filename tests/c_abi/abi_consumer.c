/*
 * A plain C consumer of libwmtp's C ABI: device buffers from the HIP
 * runtime, the hot path's calls on the default stream, no torch.  It checks
 * closed forms that hold at any length:
 *
 *   K = 0 makes every selected logit 0, so the softmax over the selected keys
 *   is uniform; with V = 1 the output is exactly 1 and the log-sum-exp is the
 *   log of the number of selected keys: ln S (full context) and
 *   ln min(S, sink + W) (windowed; ring after appending S rows; the paged
 *   pool through an identity token table; a draft-extend row t of n new
 *   rows at its own length S - n + t + 1, padding rows 0 and -inf; an fp8
 *   cache of codes 0 and 1.0 with value scale 2 gives exactly 2).
 *
 * and that malformed arguments return their status before anything is
 * enqueued.  Prints one line per check; exit status 0 when all hold.
 */
#include <hip/hip_runtime_api.h>
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

#include "wmtp.h"

#define B 2
#define HQ 16
#define HKV 2
#define D 128
#define S_MAX 70000
#define W 512
#define SINK 4
#define R_W 512
#define N_MAX 600

static int failures = 0;

static void check(int ok, const char* what) {
  printf("%s %s\n", ok ? "ok  " : "FAIL", what);
  if (!ok) failures++;
}

static void* dev_alloc(size_t bytes) {
  void* p = NULL;
  if (hipMalloc(&p, bytes) != hipSuccess) {
    printf("FAIL hipMalloc(%zu)\n", bytes);
    exit(2);
  }
  return p;
}

static void hip_ok(hipError_t e, const char* what) {
  if (e != hipSuccess) {
    printf("FAIL %s: %s\n", what, hipGetErrorString(e));
    exit(2);
  }
}

#define QMAX 3
#define WIDTH 2 /* speculation candidates */
#define DD 4    /* largest speculative depth */

/* Query rows r < nrows ([nrows, HQ, D] out, [nrows, HQ] lse): the output is
 * `value` (a bf16 word) and lse == ln(n_sel[r]) where n_sel[r] > 0; a row
 * with no keys gives 0 and -inf. */
static void check_rows(const void* out, const float* lse, const int* n_sel, int nrows, uint16_t value,
                       const char* what) {
  static uint16_t o[B * QMAX * HQ * D];
  static float l[B * QMAX * HQ];
  hip_ok(hipMemcpy(o, out, (size_t)nrows * HQ * D * 2, hipMemcpyDeviceToHost), "copy out");
  hip_ok(hipMemcpy(l, lse, (size_t)nrows * HQ * sizeof(float), hipMemcpyDeviceToHost), "copy lse");
  int values = 1, empty = 1;
  double worst = 0.0;
  for (int r = 0; r < nrows; ++r) {
    const uint16_t want = n_sel[r] > 0 ? value : 0;
    for (int i = 0; i < HQ * D; ++i) values &= o[(size_t)r * HQ * D + i] == want;
    for (int h = 0; h < HQ; ++h) {
      const float x = l[r * HQ + h];
      if (n_sel[r] > 0) {
        const double e = fabs((double)x - log((double)n_sel[r]));
        if (e > worst) worst = e;
      } else {
        empty &= isinf(x) && x < 0.0f;
      }
    }
  }
  char msg[200];
  snprintf(msg, sizeof(msg), "%s: output == 0x%04x at every kept row (0 where none)", what, (unsigned)value);
  check(values, msg);
  snprintf(msg, sizeof(msg), "%s: lse == ln(selected keys) (worst error %.2e), -inf without keys", what, worst);
  check(worst <= 1e-5 && empty, msg);
}

static void check_uniform(const void* out, const float* lse, const int n_sel[B], const char* what) {
  check_rows(out, lse, n_sel, B, 0x3F80, what);
}

int main(void) {
  check(wmtp_abi_version() == WMTP_ABI_VERSION, "library ABI version matches the header");

  const size_t row = (size_t)HKV * D * 2; /* bytes of one K or V row */
  const int lens_h[B] = {S_MAX, 300};
  void* q = dev_alloc((size_t)B * HQ * D * 2);
  void* k = dev_alloc((size_t)B * S_MAX * row);
  void* v = dev_alloc((size_t)B * S_MAX * row);
  void* out = dev_alloc((size_t)B * HQ * D * 2);
  float* lse = (float*)dev_alloc((size_t)B * HQ * sizeof(float));
  int32_t* lens = (int32_t*)dev_alloc(sizeof(lens_h));
  int32_t* err = (int32_t*)dev_alloc(sizeof(int32_t));
  hip_ok(hipMemset(q, 0, (size_t)B * HQ * D * 2), "q = 0");
  hip_ok(hipMemset(k, 0, (size_t)B * S_MAX * row), "K = 0");
  hip_ok(hipMemsetD16((hipDeviceptr_t)v, 0x3F80, (size_t)B * S_MAX * row / 2), "V = 1");
  hip_ok(hipMemcpy(lens, lens_h, sizeof(lens_h), hipMemcpyHostToDevice), "lens");
  hip_ok(hipMemset(err, 0, sizeof(int32_t)), "err = 0");

  size_t ws_bytes = wmtp_workspace_bytes(B, HQ, HKV, D, S_MAX, W, SINK, WMTP_VARIANT_FULL);
  const size_t ws_win = wmtp_workspace_bytes(B, HQ, HKV, D, S_MAX, W, SINK, WMTP_VARIANT_WINDOWED);
  const size_t ws_ring = wmtp_workspace_bytes(B, HQ, HKV, D, SINK + R_W, W, SINK, WMTP_VARIANT_RING);
  const size_t ws_ext = wmtp_workspace_bytes(B * QMAX, HQ, HKV, D, S_MAX, W, SINK, WMTP_VARIANT_WINDOWED);
  const size_t ws_pool = wmtp_workspace_bytes(B, HQ, HKV, D, S_MAX, W, SINK, WMTP_VARIANT_PAGED_WINDOWED);
  const size_t ws_tree = wmtp_workspace_bytes(B * WIDTH, HQ, HKV, D, 0, W, SINK, WMTP_VARIANT_TREE);
  /* the full-context extend's per-sequence items need more room than its rows' */
  const size_t ws_xfull = wmtp_extend_workspace_bytes(B, QMAX, HQ, HKV, D, S_MAX, W, SINK, WMTP_VARIANT_FULL);
  check(ws_xfull > wmtp_workspace_bytes(B * QMAX, HQ, HKV, D, S_MAX, W, SINK, WMTP_VARIANT_FULL),
        "wmtp_extend_workspace_bytes (full) exceeds wmtp_workspace_bytes of B * q_max rows");
  check(ws_bytes > 0 && ws_win > 0 && ws_ring > 0 && ws_ext > 0 && ws_pool > 0, "workspace sizes are positive");
  if (ws_win > ws_bytes) ws_bytes = ws_win;
  if (ws_ring > ws_bytes) ws_bytes = ws_ring;
  if (ws_ext > ws_bytes) ws_bytes = ws_ext;
  if (ws_pool > ws_bytes) ws_bytes = ws_pool;
  if (ws_tree > ws_bytes) ws_bytes = ws_tree;
  if (ws_xfull > ws_bytes) ws_bytes = ws_xfull;
  void* ws = dev_alloc(ws_bytes);
  hip_ok(hipMemset(ws, 0, ws_bytes), "workspace zero-filled once");
  const float scale = 1.0f / sqrtf((float)D);

  /* Full context: every key. */
  int st = wmtp_draft_attn_full(q, k, v, lens, out, lse, B, HQ, HKV, D, S_MAX, scale, ws, ws_bytes, err, NULL);
  check(st == WMTP_OK, "wmtp_draft_attn_full returns OK");
  hip_ok(hipDeviceSynchronize(), "full");
  const int sel_full[B] = {S_MAX, 300};
  check_uniform(out, lse, sel_full, "full context");

  /* Windowed: the sink and the last W keys (all 300 keys of the short one). */
  st = wmtp_draft_attn_windowed(q, k, v, lens, out, lse, B, HQ, HKV, D, S_MAX, W, SINK, scale, ws,
                                ws_bytes, err, NULL);
  check(st == WMTP_OK, "wmtp_draft_attn_windowed returns OK");
  hip_ok(hipDeviceSynchronize(), "windowed");
  const int sel_win[B] = {SINK + W, 300};
  check_uniform(out, lse, sel_win, "windowed");

  /* Ring: append 600 and 300 rows (K = 0, V = 1) to empty rings, attend. */
  const int n_new_h[B] = {N_MAX, 300};
  const int zero_h[B] = {0, 0};
  void* k_ring = dev_alloc((size_t)B * (SINK + R_W) * row);
  void* v_ring = dev_alloc((size_t)B * (SINK + R_W) * row);
  void* k_new = dev_alloc((size_t)B * N_MAX * row);
  void* v_new = dev_alloc((size_t)B * N_MAX * row);
  int32_t* n_new = (int32_t*)dev_alloc(sizeof(n_new_h));
  int32_t* lens_ring = (int32_t*)dev_alloc(sizeof(zero_h));
  hip_ok(hipMemset(k_new, 0, (size_t)B * N_MAX * row), "k_new = 0");
  hip_ok(hipMemsetD16((hipDeviceptr_t)v_new, 0x3F80, (size_t)B * N_MAX * row / 2), "v_new = 1");
  hip_ok(hipMemcpy(n_new, n_new_h, sizeof(n_new_h), hipMemcpyHostToDevice), "n_new");
  hip_ok(hipMemcpy(lens_ring, zero_h, sizeof(zero_h), hipMemcpyHostToDevice), "ring lens");
  st = wmtp_ring_append(k_ring, v_ring, k_new, v_new, n_new, lens_ring, B, HKV, D, SINK, R_W, N_MAX, err, NULL);
  check(st == WMTP_OK, "wmtp_ring_append returns OK");
  st = wmtp_ring_attn(q, k_ring, v_ring, lens_ring, out, lse, B, HQ, HKV, D, W, SINK, R_W, scale, ws,
                      ws_bytes, err, NULL);
  check(st == WMTP_OK, "wmtp_ring_attn returns OK");
  hip_ok(hipDeviceSynchronize(), "ring");
  int lens_after[B];
  hip_ok(hipMemcpy(lens_after, lens_ring, sizeof(lens_after), hipMemcpyDeviceToHost), "ring lens back");
  check(lens_after[0] == N_MAX && lens_after[1] == 300, "ring lengths advanced by n_new on the device");
  const int sel_ring[B] = {SINK + W, 300};
  check_uniform(out, lse, sel_ring, "ring");

  /* Paged pool: the dense cache's rows as one pool, req_to_token[b][p] = b S_MAX + p. */
  int32_t* table_h = (int32_t*)malloc(sizeof(int32_t) * B * S_MAX);
  if (table_h == NULL) return 2;
  for (int b = 0; b < B; ++b)
    for (int p = 0; p < S_MAX; ++p) table_h[b * S_MAX + p] = b * S_MAX + p;
  int32_t* table = (int32_t*)dev_alloc(sizeof(int32_t) * B * S_MAX);
  hip_ok(hipMemcpy(table, table_h, sizeof(int32_t) * B * S_MAX, hipMemcpyHostToDevice), "table");
  free(table_h);
  st = wmtp_paged_attn_windowed(q, k, v, table, lens, out, lse, B, HQ, HKV, D, (int64_t)B * S_MAX, S_MAX, W, SINK,
                                scale, ws, ws_bytes, err, NULL);
  check(st == WMTP_OK, "wmtp_paged_attn_windowed returns OK");
  hip_ok(hipDeviceSynchronize(), "paged");
  check_uniform(out, lse, sel_win, "paged windowed");

  /* Windowed draft-extend: 3 and 2 new rows (q_max 3), the third row of the
   * short sequence is padding. */
  const int n_q_h[B] = {3, 2};
  int sel_ext[B * QMAX];
  for (int b = 0; b < B; ++b)
    for (int t = 0; t < QMAX; ++t) {
      const int L = t < n_q_h[b] ? lens_h[b] - n_q_h[b] + t + 1 : 0;
      sel_ext[b * QMAX + t] = L > SINK + W ? SINK + W : L;
    }
  void* q3 = dev_alloc((size_t)B * QMAX * HQ * D * 2);
  void* out3 = dev_alloc((size_t)B * QMAX * HQ * D * 2);
  float* lse3 = (float*)dev_alloc((size_t)B * QMAX * HQ * sizeof(float));
  int32_t* n_q = (int32_t*)dev_alloc(sizeof(n_q_h));
  hip_ok(hipMemset(q3, 0, (size_t)B * QMAX * HQ * D * 2), "q3 = 0");
  hip_ok(hipMemcpy(n_q, n_q_h, sizeof(n_q_h), hipMemcpyHostToDevice), "n_q");
  st = wmtp_draft_extend_windowed(q3, k, v, lens, n_q, out3, lse3, B, QMAX, HQ, HKV, D, S_MAX, W, SINK, scale, ws,
                                  ws_bytes, err, NULL);
  check(st == WMTP_OK, "wmtp_draft_extend_windowed returns OK");
  hip_ok(hipDeviceSynchronize(), "extend");
  check_rows(out3, lse3, sel_ext, B * QMAX, 0x3F80, "windowed extend");
  /* The same rows over the full context (row t sees lens - n + t + 1 keys). */
  int sel_xfull[B * QMAX];
  for (int b = 0; b < B; ++b)
    for (int t = 0; t < QMAX; ++t) sel_xfull[b * QMAX + t] = t < n_q_h[b] ? lens_h[b] - n_q_h[b] + t + 1 : 0;
  st = wmtp_draft_extend_full(q3, k, v, lens, n_q, out3, lse3, B, QMAX, HQ, HKV, D, S_MAX, scale, ws, ws_bytes, err,
                              NULL);
  check(st == WMTP_OK, "wmtp_draft_extend_full returns OK");
  hip_ok(hipDeviceSynchronize(), "full extend");
  check_rows(out3, lse3, sel_xfull, B * QMAX, 0x3F80, "full extend");

  /* fp8 cache: K codes 0, V codes 0x38 (E4M3 1.0), value scale 2 -> output 2. */
  const size_t row8 = (size_t)HKV * D;
  void* k8 = dev_alloc((size_t)B * S_MAX * row8);
  void* v8 = dev_alloc((size_t)B * S_MAX * row8);
  hip_ok(hipMemset(k8, 0, (size_t)B * S_MAX * row8), "K codes = 0");
  hip_ok(hipMemset(v8, 0x38, (size_t)B * S_MAX * row8), "V codes = 1.0");
  st = wmtp_draft_attn_full_fp8(q, k8, v8, lens, out, lse, B, HQ, HKV, D, S_MAX, scale, 0.5f, 2.0f, ws, ws_bytes,
                                err, NULL);
  check(st == WMTP_OK, "wmtp_draft_attn_full_fp8 returns OK");
  hip_ok(hipDeviceSynchronize(), "fp8 full");
  check_rows(out, lse, sel_full, B, 0x4000, "fp8 full context");
  st = wmtp_draft_attn_windowed_fp8(q, k8, v8, lens, out, lse, B, HQ, HKV, D, S_MAX, W, SINK, scale, 0.5f, 2.0f, ws,
                                    ws_bytes, err, NULL);
  check(st == WMTP_OK, "wmtp_draft_attn_windowed_fp8 returns OK");
  hip_ok(hipDeviceSynchronize(), "fp8 windowed");
  check_rows(out, lse, sel_win, B, 0x4000, "fp8 windowed");
  st = wmtp_draft_attn_full_fp8(q, k8, v8, lens, out, lse, B, HQ, HKV, D, S_MAX, scale, 0.5f, -1.0f, ws, ws_bytes,
                                err, NULL);
  check(st == WMTP_EINVAL, "fp8 value scale -1 -> WMTP_EINVAL");

  /* Speculation: a ring of sink + W + DD slots holding 600 and 300 committed
   * rows, WIDTH candidates (candidate 1 in a private run), one draft step:
   * every candidate sees min(S + 1, sink + W) keys.  Then the depth reset
   * and a chain rollback of 5 and 7 rows. */
  const int R_WT = W + DD;
  void* kt = dev_alloc((size_t)B * (SINK + R_WT) * row);
  void* vt = dev_alloc((size_t)B * (SINK + R_WT) * row);
  void* kbr = dev_alloc((size_t)B * (WIDTH - 1) * DD * row);
  void* vbr = dev_alloc((size_t)B * (WIDTH - 1) * DD * row);
  void* q_t = dev_alloc((size_t)B * WIDTH * HQ * D * 2);
  void* out_t = dev_alloc((size_t)B * WIDTH * HQ * D * 2);
  float* lse_t = (float*)dev_alloc((size_t)B * WIDTH * HQ * sizeof(float));
  int32_t* lens_t = (int32_t*)dev_alloc(sizeof(zero_h));
  int32_t* depth = (int32_t*)dev_alloc(sizeof(zero_h));
  int32_t* n_drop = (int32_t*)dev_alloc(sizeof(zero_h));
  const int drop_h[B] = {5, 7};
  hip_ok(hipMemset(q_t, 0, (size_t)B * WIDTH * HQ * D * 2), "q_t = 0");
  hip_ok(hipMemcpy(lens_t, zero_h, sizeof(zero_h), hipMemcpyHostToDevice), "tree lens");
  hip_ok(hipMemcpy(depth, zero_h, sizeof(zero_h), hipMemcpyHostToDevice), "depth");
  hip_ok(hipMemcpy(n_drop, drop_h, sizeof(drop_h), hipMemcpyHostToDevice), "n_drop");
  st = wmtp_ring_append(kt, vt, k_new, v_new, n_new, lens_t, B, HKV, D, SINK, R_WT, N_MAX, err, NULL);
  check(st == WMTP_OK, "committed rows appended to the tree ring");
  /* the candidates' rows: the first WIDTH rows of k_new / v_new viewed as [B, WIDTH, Hkv, d] */
  st = wmtp_tree_append(kt, vt, kbr, vbr, k_new, v_new, lens_t, depth, B, WIDTH, HKV, D, W, SINK, R_WT, DD, err,
                        NULL);
  check(st == WMTP_OK, "wmtp_tree_append returns OK");
  st = wmtp_tree_attn(q_t, kt, vt, kbr, vbr, lens_t, depth, out_t, lse_t, B, WIDTH, HQ, HKV, D, W, SINK, R_WT, DD,
                      scale, ws, ws_bytes, err, NULL);
  check(st == WMTP_OK, "wmtp_tree_attn returns OK");
  hip_ok(hipDeviceSynchronize(), "tree");
  int sel_tree[B * WIDTH];
  for (int b = 0; b < B; ++b)
    for (int c = 0; c < WIDTH; ++c) sel_tree[b * WIDTH + c] = n_new_h[b] + 1 > SINK + W ? SINK + W : n_new_h[b] + 1;
  check_rows(out_t, lse_t, sel_tree, B * WIDTH, 0x3F80, "tree candidates at depth 1");
  int back[B];
  hip_ok(hipMemcpy(back, depth, sizeof(back), hipMemcpyDeviceToHost), "depth back");
  check(back[0] == 1 && back[1] == 1, "tree append advanced the depth on the device");
  st = wmtp_tree_reset(depth, B, NULL);
  check(st == WMTP_OK, "wmtp_tree_reset returns OK");
  st = wmtp_ring_rollback(lens_t, n_drop, B, err, NULL);
  check(st == WMTP_OK, "wmtp_ring_rollback returns OK");
  hip_ok(hipDeviceSynchronize(), "reset / rollback");
  hip_ok(hipMemcpy(back, depth, sizeof(back), hipMemcpyDeviceToHost), "depth back");
  check(back[0] == 0 && back[1] == 0, "depth reset to 0");
  hip_ok(hipMemcpy(back, lens_t, sizeof(back), hipMemcpyDeviceToHost), "lens back");
  check(back[0] == N_MAX - 5 && back[1] == 300 - 7, "rollback lens -= n_drop");

  /* Fused windowed draft step on the dense cache: one row appended at
   * 60000 and 300, attended at the new length in the same call. */
  const int lens_in_h[B] = {60000, 300};
  const int one_h[B] = {1, 1};
  int32_t* lens_in = (int32_t*)dev_alloc(sizeof(lens_in_h));
  int32_t* lens_out = (int32_t*)dev_alloc(sizeof(lens_in_h));
  int32_t* n_one = (int32_t*)dev_alloc(sizeof(one_h));
  hip_ok(hipMemcpy(lens_in, lens_in_h, sizeof(lens_in_h), hipMemcpyHostToDevice), "lens_in");
  hip_ok(hipMemcpy(n_one, one_h, sizeof(one_h), hipMemcpyHostToDevice), "n_one");
  st = wmtp_draft_step_windowed(q, k, v, k_new, v_new, n_one, lens_in, lens_out, out, lse, B, HQ, HKV, D, S_MAX, 1,
                                W, SINK, scale, ws, ws_bytes, err, NULL);
  check(st == WMTP_OK, "wmtp_draft_step_windowed returns OK");
  hip_ok(hipDeviceSynchronize(), "fused step");
  const int sel_step[B] = {SINK + W, 301};
  check_uniform(out, lse, sel_step, "fused windowed step");
  hip_ok(hipMemcpy(back, lens_out, sizeof(back), hipMemcpyDeviceToHost), "lens_out back");
  check(back[0] == 60001 && back[1] == 301, "fused step wrote the new lengths");

  int32_t err_h = -1;
  hip_ok(hipMemcpy(&err_h, err, sizeof(err_h), hipMemcpyDeviceToHost), "err back");
  check(err_h == 0, "no device-side error bits");

  /* Host-side argument errors: returned before anything is enqueued. */
  st = wmtp_draft_attn_windowed(q, k, v, lens, out, lse, B, HQ, HKV, D, S_MAX, 0, SINK, scale, ws,
                                ws_bytes, err, NULL);
  check(st == WMTP_EINVAL, "W = 0 -> WMTP_EINVAL");
  st = wmtp_draft_attn_full(q, k, v, lens, out, lse, B, HQ, HKV, 96, S_MAX, scale, ws, ws_bytes, err, NULL);
  check(st == WMTP_EUNSUPPORTED, "d = 96 -> WMTP_EUNSUPPORTED");
  st = wmtp_draft_attn_full(q, k, v, lens, out, lse, B, HQ, HKV, D, S_MAX, scale, ws, 0, err, NULL);
  check(st == WMTP_EWORKSPACE, "no workspace -> WMTP_EWORKSPACE");
  st = wmtp_draft_attn_full(q, k, v, lens, out, lse, B, 12, 5, D, S_MAX, scale, ws, ws_bytes, err, NULL);
  check(st == WMTP_EINVAL, "Hq not a multiple of Hkv -> WMTP_EINVAL");
  check(wmtp_status_string(WMTP_EWORKSPACE) != NULL && wmtp_status_string(WMTP_OK) != NULL,
        "status strings");

  hip_ok(hipDeviceSynchronize(), "final");
  hipFree(q); hipFree(k); hipFree(v); hipFree(out); hipFree(lse); hipFree(lens); hipFree(err); hipFree(ws);
  hipFree(k_ring); hipFree(v_ring); hipFree(k_new); hipFree(v_new); hipFree(n_new); hipFree(lens_ring);
  hipFree(table); hipFree(q3); hipFree(out3); hipFree(lse3); hipFree(n_q); hipFree(k8); hipFree(v8);
  hipFree(kt); hipFree(vt); hipFree(kbr); hipFree(vbr); hipFree(q_t); hipFree(out_t); hipFree(lse_t);
  hipFree(lens_t); hipFree(depth); hipFree(n_drop); hipFree(lens_in); hipFree(lens_out); hipFree(n_one);
  printf("%d failure(s)\n", failures);
  return failures == 0 ? 0 : 1;
}
