// C ABI of libwmtp.so: host-side validation and launch of the kernels.
// Every check runs before anything is enqueued; nothing here allocates,
// synchronises or keeps state.

#include "../../include/wmtp.h"
#include "launch.h"

#include <algorithm>
#include <atomic>
#include <climits>
#include <cmath>
#include <cstdint>
#include <mutex>

#define WMTP_EXPORT extern "C" __attribute__((visibility("default")))

namespace {

using wmtp::AttnLaunch;
using wmtp::SplitPlan;

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

// Head shape: EINVAL for malformed values, EUNSUPPORTED for well-formed
// shapes without a kernel (d not 64/128/256, more than 16 query heads per KV
// head).
int check_heads(int B, int Hq, int Hkv, int d) {
  if (B < 0 || Hkv < 1 || Hq < 1 || d < 1 || Hq % Hkv != 0) return WMTP_EINVAL;
  if (d != 64 && d != 128 && d != 256) return WMTP_EUNSUPPORTED;
  if (Hq / Hkv > 16) return WMTP_EUNSUPPORTED;
  return WMTP_OK;
}

int check_window(int W, int sink) {
  if (W < 1 || sink < 0 || static_cast<int64_t>(W) + sink > INT_MAX / 2) return WMTP_EINVAL;
  return WMTP_OK;
}

// Most keys one sequence attends, for the split plan.  The windowed and ring
// variants plan for sink + W whatever the cache capacity, so both split the
// same key set identically (bit-identical results).
int64_t keys_max(int variant, int64_t S_max, int W, int sink) {
  return (variant == WMTP_VARIANT_FULL || variant == WMTP_VARIANT_PAGED_FULL)
             ? S_max
             : static_cast<int64_t>(W) + sink;
}

bool windowed_variant(int variant) {
  return variant == WMTP_VARIANT_WINDOWED || variant == WMTP_VARIANT_RING ||
         variant == WMTP_VARIANT_PAGED_WINDOWED || variant == WMTP_VARIANT_TREE;
}

bool paged_variant(int variant) {
  return variant == WMTP_VARIANT_PAGED_FULL || variant == WMTP_VARIANT_PAGED_WINDOWED;
}

// Whether a call takes the one-launch kernel (split, ticket and merge in
// one launch): windowed calls of at most kWinOneLaunchRows query rows x KV
// heads, and full-context calls of that size over a short cache (up to
// kWinFullMaxKeys rows per sequence at d = 256, a quarter of that below:
// launch-bound like the windowed ones).  The keys it plans for: the window,
// or the capacity.
bool one_launch(int variant, int rows_q, int Hkv, int d, int64_t S_max) {
  if (windowed_variant(variant)) return wmtp::use_window_kernel(rows_q, Hkv);
  if (variant == WMTP_VARIANT_FULL || variant == WMTP_VARIANT_PAGED_FULL)
    return wmtp::use_window_kernel_full(rows_q, Hkv, d, S_max);
  return false;
}
int one_launch_keys(int variant, int64_t S_max, int W, int sink) {
  return windowed_variant(variant) ? W + sink : static_cast<int>(S_max);
}

// A per-tensor scale of an fp8 cache: finite and positive.
bool valid_scale(float s) { return std::isfinite(s) && s > 0.0f; }

bool plan_fits(const SplitPlan& p, int Hkv) {
  return static_cast<int64_t>(p.max_items) * Hkv < INT_MAX;
}

// The windowed kernel's work items (and their workgroups, eight per group
// of eight items per slice) must be countable in an int.
bool win_plan_fits(const wmtp::WinPlan& p, int64_t NV, int Hkv) {
  const int64_t items = NV * Hkv * p.n_items;
  return p.n_items > 0 && NV * Hkv * p.slices <= wmtp::kMaxTickets &&
         (items + 7) / 8 * 8 * p.slices < INT_MAX / 2;
}

// Largest number of query rows per sequence an extend call accepts.
constexpr int kMaxQueryRows = 4096;

// S_max: dense rows per sequence / ring slots / request-table capacity.
// pool_rows: rows of the shared pool (paged variants only).
int attention_common(int variant, const void* q, const void* k, const void* v,
                     const int32_t* lens, const int32_t* n_q, int q_max, void* out, float* lse,
                     int B, int Hq, int Hkv, int d, int64_t S_max, int W, int sink, int R_w,
                     float scale, void* ws, size_t ws_bytes, int32_t* err, hipStream_t stream,
                     const int32_t* table = nullptr, int64_t pool_rows = 0, bool fp8 = false,
                     float k_scale = 1.0f, float v_scale = 1.0f, const void* k2 = nullptr,
                     const void* v2 = nullptr, int dd = 0, bool step = false,
                     int32_t* lens_out = nullptr, bool dry_run = false, bool check_ws = true) {
  int st = check_heads(B, Hq, Hkv, d);
  if (st != WMTP_OK) return st;
  const bool tree = variant == WMTP_VARIANT_TREE;
  // Tree: q_max candidates per request; the ring's window region holds the
  // window plus the draft-extend headroom (R_w >= W + dd), candidates 1 ..
  // q_max - 1 own private runs of dd rows.  Fused step: k2 / v2 hold the
  // dd = n_max new rows per sequence.
  const int64_t rows2 = tree ? static_cast<int64_t>(q_max - 1) * dd : (step ? dd : 0);
  if (step) {
    if (fp8 || tree || paged_variant(variant) || variant == WMTP_VARIANT_FULL || q_max != 1 || dd < 0)
      return WMTP_EINVAL;
    if (variant != WMTP_VARIANT_RING && S_max + dd > INT_MAX) return WMTP_EINVAL;
  }
  if (tree) {
    if (fp8 || dd < 1 || q_max < 1) return WMTP_EINVAL;
    if (static_cast<int64_t>(R_w) < static_cast<int64_t>(W) + dd) return WMTP_EINVAL;
    if (static_cast<int64_t>(sink) + R_w + rows2 > INT_MAX) return WMTP_EINVAL;
  }
  if (fp8 && (!valid_scale(k_scale) || !valid_scale(v_scale))) return WMTP_EINVAL;
  if (q_max < 1 || q_max > kMaxQueryRows) return WMTP_EINVAL;
  if (static_cast<int64_t>(B) * q_max > INT_MAX / 64) return WMTP_EINVAL;
  if (windowed_variant(variant)) {
    st = check_window(W, sink);
    if (st != WMTP_OK) return st;
  }
  if (paged_variant(variant) && (pool_rows < 1 || pool_rows > INT_MAX)) return WMTP_EINVAL;
  // The ring must hold the window of the earliest new row as well.
  if (variant == WMTP_VARIANT_RING && static_cast<int64_t>(R_w) < static_cast<int64_t>(W) + q_max - 1)
    return WMTP_EINVAL;
  if (S_max < 0) return WMTP_EINVAL;
  if (!std::isfinite(scale) || !std::isfinite(scale * k_scale)) return WMTP_EINVAL;
  if (B == 0) return WMTP_OK;
  if (q == nullptr || k == nullptr || v == nullptr || lens == nullptr || out == nullptr)
    return WMTP_EINVAL;
  if (paged_variant(variant) && (table == nullptr || !aligned(table, 4))) return WMTP_EINVAL;
  if ((tree || step) && (n_q == nullptr || (rows2 > 0 && (k2 == nullptr || v2 == nullptr ||
                                                           !aligned(k2, 16) || !aligned(v2, 16)))))
    return WMTP_EINVAL;
  if (step && (lens_out == nullptr || !aligned(lens_out, 4) || lens_out == lens)) return WMTP_EINVAL;
  if (!aligned(q, 16) || !aligned(k, 16) || !aligned(v, 16) || !aligned(out, 16) ||
      !aligned(lens, 4) || (lse != nullptr && !aligned(lse, 4)) ||
      (err != nullptr && !aligned(err, 4)) || (n_q != nullptr && !aligned(n_q, 4)))
    return WMTP_EINVAL;

  const int rows_q = B * q_max;
  const bool win = one_launch(variant, rows_q, Hkv, d, S_max);
  SplitPlan plan{};
  wmtp::WinPlan wp{};
  size_t need = 0;
  bool per_seq = false;
  if (win) {
    wp = wmtp::plan_window(rows_q, Hq, Hkv, d, one_launch_keys(variant, S_max, W, sink));
    if (!win_plan_fits(wp, rows_q, Hkv)) return WMTP_EUNSUPPORTED;
    need = wp.bytes;
  } else {
    plan = wmtp::plan_split(variant, rows_q, Hq, Hkv, d, keys_max(variant, S_max, W, sink));
    if (!plan_fits(plan, Hkv)) return WMTP_EUNSUPPORTED;
    need = plan.bytes;
    // A full-context extend whose workspace also holds the finer per-sequence
    // decomposition (wmtp_extend_workspace_bytes) spreads each sequence's
    // keys over about one workgroup per CU however many rows it has.
    if (variant == WMTP_VARIANT_FULL && q_max > 1 && check_ws && wmtp::rows_kernel_fits(Hkv, d, fp8)) {
      const SplitPlan fine = wmtp::plan_split(variant, rows_q, Hq, Hkv, d, keys_max(variant, S_max, W, sink), q_max);
      if (plan_fits(fine, Hkv) && ws_bytes >= fine.bytes) {
        plan = fine;
        need = fine.bytes;
        per_seq = true;
      }
    }
  }
  if (check_ws) {
    if (ws_bytes < need) return WMTP_EWORKSPACE;
    if (need > 0 && (ws == nullptr || !aligned(ws, 256))) return WMTP_EINVAL;
  }

  AttnLaunch L{};
  L.variant = variant;
  L.kv_fp8 = fp8;
  L.q = static_cast<const uint16_t*>(q);
  L.k = k;
  L.v = v;
  L.lens = lens;
  L.n_q = n_q;
  L.qps = q_max;
  L.out = static_cast<uint16_t*>(out);
  L.lse = lse;
  L.err = err;
  L.B = B;
  L.Hq = Hq;
  L.Hkv = Hkv;
  L.d = d;
  L.table = table;
  L.table_stride = S_max;
  L.k2 = k2;
  L.v2 = v2;
  L.rows2 = rows2;
  L.dd = dd;
  L.step = step;
  L.lens_out = lens_out;
  if (variant == WMTP_VARIANT_RING || tree) {
    L.rows = static_cast<int64_t>(sink) + R_w;
    L.len_cap = INT_MAX;
  } else if (paged_variant(variant)) {
    L.rows = pool_rows;
    L.len_cap = S_max < INT_MAX ? S_max : INT_MAX;
  } else {
    L.rows = S_max;
    L.len_cap = S_max < INT_MAX ? S_max : INT_MAX;
  }
  L.W = W;
  L.sink = sink;
  L.R_w = R_w;
  L.scale = scale;
  L.k_scale = k_scale;
  L.v_scale = v_scale;
  L.per_seq = per_seq;
  L.target = plan.target;
  L.chunk_cap = plan.chunk_cap;
  L.max_items = plan.max_items;
  L.win_keys = wp.item_keys;
  L.win_items = wp.n_items;
  L.win_slices = wp.slices;
  if (dry_run) return WMTP_OK;
  char* base = static_cast<char*>(ws);
  L.tickets = reinterpret_cast<int32_t*>(base);
  L.pm = reinterpret_cast<float*>(base + (win ? wp.off_pm : plan.off_pm));
  L.pl = reinterpret_cast<float*>(base + (win ? wp.off_pl : plan.off_pl));
  L.pz = reinterpret_cast<float*>(base + (win ? wp.off_pz : plan.off_pz));
  L.po = reinterpret_cast<float*>(base + (win ? wp.off_po : plan.off_po));
  if (wmtp::launch_attention(L, stream) != hipSuccess)
    return WMTP_ELAUNCH;
  return WMTP_OK;
}

int append_common(bool ring, void* k, void* v, const void* k_new, const void* v_new,
                  const int32_t* n_new, int32_t* lens, int B, int Hkv, int d, int64_t rows,
                  int sink, int R_w, int n_max, int32_t* err, hipStream_t stream, bool fp8 = false,
                  float k_scale = 1.0f, float v_scale = 1.0f, int32_t* lens_out = nullptr,
                  bool dry_run = false) {
  if (B < 0 || Hkv < 1 || d < 1 || n_max < 0) return WMTP_EINVAL;
  if (fp8 && (!valid_scale(k_scale) || !valid_scale(v_scale))) return WMTP_EINVAL;
  if (d != 64 && d != 128 && d != 256) return WMTP_EUNSUPPORTED;
  if (ring && (sink < 0 || R_w < 1 || static_cast<int64_t>(sink) + R_w > INT_MAX))
    return WMTP_EINVAL;
  if (!ring && (rows < 0 || rows > INT_MAX)) return WMTP_EINVAL;
  if (B == 0) return WMTP_OK;
  if (k == nullptr || v == nullptr || lens == nullptr || n_new == nullptr) return WMTP_EINVAL;
  if (n_max > 0 && (k_new == nullptr || v_new == nullptr)) return WMTP_EINVAL;
  if (!aligned(k, 16) || !aligned(v, 16) || !aligned(k_new, 16) || !aligned(v_new, 16) ||
      !aligned(n_new, 4) || !aligned(lens, 4) || (err != nullptr && !aligned(err, 4)) ||
      (lens_out != nullptr && (!aligned(lens_out, 4) || lens_out == lens)))
    return WMTP_EINVAL;
  if (dry_run) return WMTP_OK;
  wmtp::AppendLaunch L{};
  L.ring = ring;
  L.fp8 = fp8;
  L.k_scale = k_scale;
  L.v_scale = v_scale;
  L.k = k;
  L.v = v;
  L.k_new = static_cast<const uint16_t*>(k_new);
  L.v_new = static_cast<const uint16_t*>(v_new);
  L.n_new = n_new;
  L.lens = lens;
  L.err = err;
  L.B = B;
  L.Hkv = Hkv;
  L.d = d;
  L.rows = ring ? static_cast<int64_t>(sink) + R_w : rows;
  L.sink = ring ? sink : 0;
  L.R_w = ring ? R_w : 1;
  L.n_max = n_max;
  L.lens_out = lens_out;
  if (wmtp::launch_append(L, stream) != hipSuccess) return WMTP_ELAUNCH;
  return WMTP_OK;
}

}  // namespace

WMTP_EXPORT size_t wmtp_workspace_bytes(int B, int Hq, int Hkv, int d, int64_t S_max, int W,
                                        int sink, int variant) {
  if (variant < WMTP_VARIANT_FULL || variant > WMTP_VARIANT_TREE) return 0;
  if (check_heads(B, Hq, Hkv, d) != WMTP_OK || B == 0) return 0;
  if (windowed_variant(variant) && check_window(W, sink) != WMTP_OK) return 0;
  if (!windowed_variant(variant) && S_max < 0) return 0;
  if (one_launch(variant, B, Hkv, d, S_max)) {
    const wmtp::WinPlan wp = wmtp::plan_window(B, Hq, Hkv, d, one_launch_keys(variant, S_max, W, sink));
    if (!win_plan_fits(wp, B, Hkv)) return 0;
    return wp.bytes;
  }
  const SplitPlan plan =
      wmtp::plan_split(variant, B, Hq, Hkv, d, keys_max(variant, S_max, W, sink));
  if (!plan_fits(plan, Hkv)) return 0;
  return plan.bytes;
}

WMTP_EXPORT size_t wmtp_extend_workspace_bytes(int B, int q_max, int Hq, int Hkv, int d, int64_t S_max,
                                               int W, int sink, int variant) {
  if (B < 0 || q_max < 1 || q_max > kMaxQueryRows || static_cast<int64_t>(B) * q_max > INT_MAX / 64) return 0;
  const int rows_q = B * q_max;
  const size_t coarse = wmtp_workspace_bytes(rows_q, Hq, Hkv, d, S_max, W, sink, variant);
  if (variant != WMTP_VARIANT_FULL || q_max == 1 || coarse == 0) return coarse;
  const SplitPlan fine = wmtp::plan_split(variant, rows_q, Hq, Hkv, d, keys_max(variant, S_max, W, sink), q_max);
  return plan_fits(fine, Hkv) ? std::max(coarse, fine.bytes) : coarse;
}

WMTP_EXPORT int wmtp_draft_attn_full(const void* q, const void* k, const void* v,
                                     const int32_t* lens, void* out, float* lse, int B, int Hq,
                                     int Hkv, int d, int64_t S_max, float scale, void* ws,
                                     size_t ws_bytes, int32_t* err, hipStream_t stream) {
  return attention_common(WMTP_VARIANT_FULL, q, k, v, lens, nullptr, 1, out, lse, B, Hq, Hkv, d,
                          S_max, 1, 0, 1, scale, ws, ws_bytes, err, stream);
}

WMTP_EXPORT int wmtp_draft_attn_windowed(const void* q, const void* k, const void* v,
                                         const int32_t* lens, void* out, float* lse, int B,
                                         int Hq, int Hkv, int d, int64_t S_max, int W, int sink,
                                         float scale, void* ws, size_t ws_bytes, int32_t* err,
                                         hipStream_t stream) {
  return attention_common(WMTP_VARIANT_WINDOWED, q, k, v, lens, nullptr, 1, out, lse, B, Hq, Hkv,
                          d, S_max, W, sink, W, scale, ws, ws_bytes, err, stream);
}

WMTP_EXPORT int wmtp_ring_attn(const void* q, const void* k_ring, const void* v_ring,
                               const int32_t* lens, void* out, float* lse, int B, int Hq, int Hkv,
                               int d, int W, int sink, int R_w, float scale, void* ws,
                               size_t ws_bytes, int32_t* err, hipStream_t stream) {
  if (check_window(W, sink) == WMTP_OK && (R_w < W || static_cast<int64_t>(sink) + R_w > INT_MAX))
    return WMTP_EINVAL;
  return attention_common(WMTP_VARIANT_RING, q, k_ring, v_ring, lens, nullptr, 1, out, lse, B, Hq,
                          Hkv, d, static_cast<int64_t>(sink) + R_w, W, sink, R_w, scale, ws,
                          ws_bytes, err, stream);
}

WMTP_EXPORT int wmtp_draft_extend_full(const void* q, const void* k, const void* v,
                                       const int32_t* lens, const int32_t* n_q, void* out,
                                       float* lse, int B, int q_max, int Hq, int Hkv, int d,
                                       int64_t S_max, float scale, void* ws, size_t ws_bytes,
                                       int32_t* err, hipStream_t stream) {
  return attention_common(WMTP_VARIANT_FULL, q, k, v, lens, n_q, q_max, out, lse, B, Hq, Hkv, d,
                          S_max, 1, 0, 1, scale, ws, ws_bytes, err, stream);
}

WMTP_EXPORT int wmtp_draft_extend_windowed(const void* q, const void* k, const void* v,
                                           const int32_t* lens, const int32_t* n_q, void* out,
                                           float* lse, int B, int q_max, int Hq, int Hkv, int d,
                                           int64_t S_max, int W, int sink, float scale, void* ws,
                                           size_t ws_bytes, int32_t* err, hipStream_t stream) {
  return attention_common(WMTP_VARIANT_WINDOWED, q, k, v, lens, n_q, q_max, out, lse, B, Hq, Hkv,
                          d, S_max, W, sink, W, scale, ws, ws_bytes, err, stream);
}

WMTP_EXPORT int wmtp_ring_extend(const void* q, const void* k_ring, const void* v_ring,
                                 const int32_t* lens, const int32_t* n_q, void* out, float* lse,
                                 int B, int q_max, int Hq, int Hkv, int d, int W, int sink,
                                 int R_w, float scale, void* ws, size_t ws_bytes, int32_t* err,
                                 hipStream_t stream) {
  if (check_window(W, sink) == WMTP_OK && static_cast<int64_t>(sink) + R_w > INT_MAX)
    return WMTP_EINVAL;
  return attention_common(WMTP_VARIANT_RING, q, k_ring, v_ring, lens, n_q, q_max, out, lse, B, Hq,
                          Hkv, d, static_cast<int64_t>(sink) + R_w, W, sink, R_w, scale, ws,
                          ws_bytes, err, stream);
}

WMTP_EXPORT int wmtp_paged_attn_full(const void* q, const void* k_pool, const void* v_pool,
                                      const int32_t* req_to_token, const int32_t* lens, void* out,
                                      float* lse, int B, int Hq, int Hkv, int d, int64_t pool_rows,
                                      int64_t table_stride, float scale, void* ws, size_t ws_bytes,
                                      int32_t* err, hipStream_t stream) {
  return attention_common(WMTP_VARIANT_PAGED_FULL, q, k_pool, v_pool, lens, nullptr, 1, out, lse, B,
                          Hq, Hkv, d, table_stride, 1, 0, 1, scale, ws, ws_bytes, err, stream,
                          req_to_token, pool_rows);
}

WMTP_EXPORT int wmtp_paged_attn_windowed(const void* q, const void* k_pool, const void* v_pool,
                                          const int32_t* req_to_token, const int32_t* lens,
                                          void* out, float* lse, int B, int Hq, int Hkv, int d,
                                          int64_t pool_rows, int64_t table_stride, int W, int sink,
                                          float scale, void* ws, size_t ws_bytes, int32_t* err,
                                          hipStream_t stream) {
  return attention_common(WMTP_VARIANT_PAGED_WINDOWED, q, k_pool, v_pool, lens, nullptr, 1, out,
                          lse, B, Hq, Hkv, d, table_stride, W, sink, W, scale, ws, ws_bytes, err,
                          stream, req_to_token, pool_rows);
}

WMTP_EXPORT int64_t wmtp_kv_indices_capacity(int variant, int B, int64_t table_stride, int W,
                                             int sink) {
  if (B < 0 || table_stride < 0) return 0;
  if (variant != WMTP_VARIANT_PAGED_FULL && variant != WMTP_VARIANT_PAGED_WINDOWED) return 0;
  if (variant == WMTP_VARIANT_PAGED_WINDOWED && check_window(W, sink) != WMTP_OK) return 0;
  const int64_t per = variant == WMTP_VARIANT_PAGED_FULL
                          ? table_stride
                          : std::min<int64_t>(table_stride, static_cast<int64_t>(W) + sink);
  return static_cast<int64_t>(B) * per;
}

WMTP_EXPORT int wmtp_build_kv_indices(const int32_t* req_to_token, const int32_t* lens, int B,
                                      int64_t table_stride, int variant, int W, int sink,
                                      int32_t* kv_indptr, int32_t* kv_indices, int64_t capacity,
                                      int32_t* err, hipStream_t stream) {
  if (B < 0 || B > 65535 || table_stride < 0 || table_stride > INT_MAX) return WMTP_EINVAL;
  if (variant != WMTP_VARIANT_PAGED_FULL && variant != WMTP_VARIANT_PAGED_WINDOWED)
    return WMTP_EINVAL;
  const bool windowed = variant == WMTP_VARIANT_PAGED_WINDOWED;
  if (windowed && check_window(W, sink) != WMTP_OK) return WMTP_EINVAL;
  if (capacity < wmtp_kv_indices_capacity(variant, B, table_stride, W, sink)) return WMTP_EWORKSPACE;
  if (capacity > INT_MAX) return WMTP_EUNSUPPORTED;  // int32 offsets in kv_indptr
  if (B == 0) return WMTP_OK;
  if (req_to_token == nullptr || lens == nullptr || kv_indptr == nullptr ||
      (capacity > 0 && kv_indices == nullptr))
    return WMTP_EINVAL;
  if (!aligned(req_to_token, 4) || !aligned(lens, 4) || !aligned(kv_indptr, 4) ||
      !aligned(kv_indices, 4) || (err != nullptr && !aligned(err, 4)))
    return WMTP_EINVAL;
  const int64_t n_keys_max = windowed ? std::min<int64_t>(table_stride, static_cast<int64_t>(W) + sink)
                                      : table_stride;
  if (wmtp::launch_kv_indices(req_to_token, table_stride, lens, B, windowed, W, sink, n_keys_max,
                              kv_indptr, kv_indices, err,
                              stream) != hipSuccess)
    return WMTP_ELAUNCH;
  return WMTP_OK;
}

WMTP_EXPORT int wmtp_ring_append(void* k_ring, void* v_ring, const void* k_new,
                                 const void* v_new, const int32_t* n_new, int32_t* lens, int B,
                                 int Hkv, int d, int sink, int R_w, int n_max, int32_t* err,
                                 hipStream_t stream) {
  return append_common(true, k_ring, v_ring, k_new, v_new, n_new, lens, B, Hkv, d, 0, sink, R_w,
                       n_max, err, stream);
}

WMTP_EXPORT int wmtp_cache_append(void* k, void* v, const void* k_new, const void* v_new,
                                  const int32_t* n_new, int32_t* lens, int B, int Hkv, int d,
                                  int64_t S_max, int n_max, int32_t* err, hipStream_t stream) {
  return append_common(false, k, v, k_new, v_new, n_new, lens, B, Hkv, d, S_max, 0, 1, n_max, err,
                       stream);
}

WMTP_EXPORT int wmtp_draft_attn_full_fp8(const void* q, const void* k, const void* v,
                                         const int32_t* lens, void* out, float* lse, int B, int Hq,
                                         int Hkv, int d, int64_t S_max, float scale, float k_scale,
                                         float v_scale, void* ws, size_t ws_bytes, int32_t* err,
                                         hipStream_t stream) {
  return attention_common(WMTP_VARIANT_FULL, q, k, v, lens, nullptr, 1, out, lse, B, Hq, Hkv, d,
                          S_max, 1, 0, 1, scale, ws, ws_bytes, err, stream, nullptr, 0, true,
                          k_scale, v_scale);
}

WMTP_EXPORT int wmtp_draft_attn_windowed_fp8(const void* q, const void* k, const void* v,
                                             const int32_t* lens, void* out, float* lse, int B,
                                             int Hq, int Hkv, int d, int64_t S_max, int W, int sink,
                                             float scale, float k_scale, float v_scale, void* ws,
                                             size_t ws_bytes, int32_t* err, hipStream_t stream) {
  return attention_common(WMTP_VARIANT_WINDOWED, q, k, v, lens, nullptr, 1, out, lse, B, Hq, Hkv,
                          d, S_max, W, sink, W, scale, ws, ws_bytes, err, stream, nullptr, 0, true,
                          k_scale, v_scale);
}

WMTP_EXPORT int wmtp_draft_extend_full_fp8(const void* q, const void* k, const void* v,
                                           const int32_t* lens, const int32_t* n_q, void* out,
                                           float* lse, int B, int q_max, int Hq, int Hkv, int d,
                                           int64_t S_max, float scale, float k_scale, float v_scale,
                                           void* ws, size_t ws_bytes, int32_t* err, hipStream_t stream) {
  return attention_common(WMTP_VARIANT_FULL, q, k, v, lens, n_q, q_max, out, lse, B, Hq, Hkv, d,
                          S_max, 1, 0, 1, scale, ws, ws_bytes, err, stream, nullptr, 0, true,
                          k_scale, v_scale);
}

WMTP_EXPORT int wmtp_draft_extend_windowed_fp8(const void* q, const void* k, const void* v,
                                               const int32_t* lens, const int32_t* n_q, void* out,
                                               float* lse, int B, int q_max, int Hq, int Hkv,
                                               int d, int64_t S_max, int W, int sink, float scale,
                                               float k_scale, float v_scale, void* ws,
                                               size_t ws_bytes, int32_t* err, hipStream_t stream) {
  return attention_common(WMTP_VARIANT_WINDOWED, q, k, v, lens, n_q, q_max, out, lse, B, Hq, Hkv,
                          d, S_max, W, sink, W, scale, ws, ws_bytes, err, stream, nullptr, 0, true,
                          k_scale, v_scale);
}

WMTP_EXPORT int wmtp_ring_extend_fp8(const void* q, const void* k_ring, const void* v_ring,
                                     const int32_t* lens, const int32_t* n_q, void* out,
                                     float* lse, int B, int q_max, int Hq, int Hkv, int d, int W,
                                     int sink, int R_w, float scale, float k_scale, float v_scale,
                                     void* ws, size_t ws_bytes, int32_t* err, hipStream_t stream) {
  if (check_window(W, sink) == WMTP_OK && static_cast<int64_t>(sink) + R_w > INT_MAX)
    return WMTP_EINVAL;
  return attention_common(WMTP_VARIANT_RING, q, k_ring, v_ring, lens, n_q, q_max, out, lse, B, Hq,
                          Hkv, d, static_cast<int64_t>(sink) + R_w, W, sink, R_w, scale, ws,
                          ws_bytes, err, stream, nullptr, 0, true, k_scale, v_scale);
}

WMTP_EXPORT int wmtp_paged_attn_full_fp8(const void* q, const void* k_pool, const void* v_pool,
                                          const int32_t* req_to_token, const int32_t* lens, void* out,
                                          float* lse, int B, int Hq, int Hkv, int d, int64_t pool_rows,
                                          int64_t table_stride, float scale, float k_scale,
                                          float v_scale, void* ws, size_t ws_bytes, int32_t* err,
                                          hipStream_t stream) {
  return attention_common(WMTP_VARIANT_PAGED_FULL, q, k_pool, v_pool, lens, nullptr, 1, out, lse, B,
                          Hq, Hkv, d, table_stride, 1, 0, 1, scale, ws, ws_bytes, err, stream,
                          req_to_token, pool_rows, true, k_scale, v_scale);
}

WMTP_EXPORT int wmtp_paged_attn_windowed_fp8(const void* q, const void* k_pool, const void* v_pool,
                                              const int32_t* req_to_token, const int32_t* lens,
                                              void* out, float* lse, int B, int Hq, int Hkv, int d,
                                              int64_t pool_rows, int64_t table_stride, int W,
                                              int sink, float scale, float k_scale, float v_scale,
                                              void* ws, size_t ws_bytes, int32_t* err, hipStream_t stream) {
  return attention_common(WMTP_VARIANT_PAGED_WINDOWED, q, k_pool, v_pool, lens, nullptr, 1, out,
                          lse, B, Hq, Hkv, d, table_stride, W, sink, W, scale, ws, ws_bytes, err,
                          stream, req_to_token, pool_rows, true, k_scale, v_scale);
}

WMTP_EXPORT int wmtp_ring_attn_fp8(const void* q, const void* k_ring, const void* v_ring,
                                   const int32_t* lens, void* out, float* lse, int B, int Hq,
                                   int Hkv, int d, int W, int sink, int R_w, float scale,
                                   float k_scale, float v_scale, void* ws, size_t ws_bytes,
                                   int32_t* err, hipStream_t stream) {
  if (check_window(W, sink) == WMTP_OK && (R_w < W || static_cast<int64_t>(sink) + R_w > INT_MAX))
    return WMTP_EINVAL;
  return attention_common(WMTP_VARIANT_RING, q, k_ring, v_ring, lens, nullptr, 1, out, lse, B, Hq,
                          Hkv, d, static_cast<int64_t>(sink) + R_w, W, sink, R_w, scale, ws,
                          ws_bytes, err, stream, nullptr, 0, true, k_scale, v_scale);
}

WMTP_EXPORT int wmtp_ring_append_fp8(void* k_ring, void* v_ring, const void* k_new,
                                     const void* v_new, const int32_t* n_new, int32_t* lens, int B,
                                     int Hkv, int d, int sink, int R_w, int n_max, float k_scale,
                                     float v_scale, int32_t* err, hipStream_t stream) {
  return append_common(true, k_ring, v_ring, k_new, v_new, n_new, lens, B, Hkv, d, 0, sink, R_w,
                       n_max, err, stream, true, k_scale, v_scale);
}

WMTP_EXPORT int wmtp_cache_append_fp8(void* k, void* v, const void* k_new, const void* v_new,
                                      const int32_t* n_new, int32_t* lens, int B, int Hkv, int d,
                                      int64_t S_max, int n_max, float k_scale, float v_scale,
                                      int32_t* err, hipStream_t stream) {
  return append_common(false, k, v, k_new, v_new, n_new, lens, B, Hkv, d, S_max, 0, 1, n_max, err,
                       stream, true, k_scale, v_scale);
}

WMTP_EXPORT int wmtp_draft_step_full(const void* q, void* k, void* v, const void* k_new,
                                     const void* v_new, const int32_t* n_new,
                                     const int32_t* lens_in, int32_t* lens_out, void* out,
                                     float* lse, int B, int Hq, int Hkv, int d, int64_t S_max,
                                     int n_max, float scale, void* ws, size_t ws_bytes,
                                     int32_t* err, hipStream_t stream) {
  // The full-context step is the append (lens_in -> lens_out) followed by the
  // full attention at lens_out: reading the new rows through the fused path
  // costs the O(S) kernel more than the separate append launch saves.
  if (B > 0 && (lens_in == nullptr || lens_out == nullptr)) return WMTP_EINVAL;
  int32_t* lin = const_cast<int32_t*>(lens_in);
  int st = append_common(false, k, v, k_new, v_new, n_new, lin, B, Hkv, d, S_max, 0, 1, n_max, err,
                         stream, false, 1.0f, 1.0f, lens_out, true);
  if (st != WMTP_OK) return st;
  st = attention_common(WMTP_VARIANT_FULL, q, k, v, lens_out, nullptr, 1, out, lse, B, Hq, Hkv, d,
                        S_max, 1, 0, 1, scale, ws, ws_bytes, err, stream, nullptr, 0, false, 1.0f,
                        1.0f, nullptr, nullptr, 0, false, nullptr, true);
  if (st != WMTP_OK) return st;
  st = append_common(false, k, v, k_new, v_new, n_new, lin, B, Hkv, d, S_max, 0, 1, n_max, err, stream,
                     false, 1.0f, 1.0f, lens_out);
  if (st != WMTP_OK) return st;
  return attention_common(WMTP_VARIANT_FULL, q, k, v, lens_out, nullptr, 1, out, lse, B, Hq, Hkv, d,
                          S_max, 1, 0, 1, scale, ws, ws_bytes, err, stream);
}

WMTP_EXPORT int wmtp_draft_step_windowed(const void* q, void* k, void* v, const void* k_new,
                                         const void* v_new, const int32_t* n_new,
                                         const int32_t* lens_in, int32_t* lens_out, void* out,
                                         float* lse, int B, int Hq, int Hkv, int d, int64_t S_max,
                                         int n_max, int W, int sink, float scale, void* ws,
                                         size_t ws_bytes, int32_t* err, hipStream_t stream) {
  return attention_common(WMTP_VARIANT_WINDOWED, q, k, v, lens_in, n_new, 1, out, lse, B, Hq, Hkv,
                          d, S_max, W, sink, W, scale, ws, ws_bytes, err, stream, nullptr, 0, false,
                          1.0f, 1.0f, k_new, v_new, n_max, true, lens_out);
}

WMTP_EXPORT int wmtp_ring_step(const void* q, void* k_ring, void* v_ring, const void* k_new,
                               const void* v_new, const int32_t* n_new, const int32_t* lens_in,
                               int32_t* lens_out, void* out, float* lse, int B, int Hq, int Hkv,
                               int d, int W, int sink, int R_w, int n_max, float scale, void* ws,
                               size_t ws_bytes, int32_t* err, hipStream_t stream) {
  if (check_window(W, sink) == WMTP_OK && (R_w < W || static_cast<int64_t>(sink) + R_w > INT_MAX))
    return WMTP_EINVAL;
  return attention_common(WMTP_VARIANT_RING, q, k_ring, v_ring, lens_in, n_new, 1, out, lse, B, Hq,
                          Hkv, d, static_cast<int64_t>(sink) + R_w, W, sink, R_w, scale, ws,
                          ws_bytes, err, stream, nullptr, 0, false, 1.0f, 1.0f, k_new, v_new, n_max,
                          true, lens_out);
}

WMTP_EXPORT int wmtp_tree_attn(const void* q, const void* k_ring, const void* v_ring,
                               const void* k_branch, const void* v_branch, const int32_t* lens,
                               const int32_t* depth, void* out, float* lse, int B, int width, int Hq,
                               int Hkv, int d, int W, int sink, int R_w, int depth_max, float scale,
                               void* ws, size_t ws_bytes, int32_t* err, hipStream_t stream) {
  return attention_common(WMTP_VARIANT_TREE, q, k_ring, v_ring, lens, depth, width, out, lse, B, Hq,
                          Hkv, d, static_cast<int64_t>(sink) + R_w, W, sink, R_w, scale, ws,
                          ws_bytes, err, stream, nullptr, 0, false, 1.0f, 1.0f, k_branch, v_branch,
                          depth_max);
}

WMTP_EXPORT int wmtp_tree_append(void* k_ring, void* v_ring, void* k_branch, void* v_branch,
                                 const void* k_new, const void* v_new, const int32_t* lens,
                                 int32_t* depth, int B, int width, int Hkv, int d, int W, int sink,
                                 int R_w, int depth_max, int32_t* err, hipStream_t stream) {
  if (B < 0 || width < 1 || Hkv < 1 || d < 1 || depth_max < 1 || sink < 0 || check_window(W, sink))
    return WMTP_EINVAL;
  if (d != 64 && d != 128 && d != 256) return WMTP_EUNSUPPORTED;
  if (static_cast<int64_t>(R_w) < static_cast<int64_t>(W) + depth_max ||
      static_cast<int64_t>(sink) + R_w + static_cast<int64_t>(width - 1) * depth_max > INT_MAX)
    return WMTP_EINVAL;
  if (B == 0) return WMTP_OK;
  if (k_ring == nullptr || v_ring == nullptr || k_new == nullptr || v_new == nullptr ||
      lens == nullptr || depth == nullptr)
    return WMTP_EINVAL;
  if (width > 1 && (k_branch == nullptr || v_branch == nullptr || !aligned(k_branch, 16) ||
                    !aligned(v_branch, 16)))
    return WMTP_EINVAL;
  if (!aligned(k_ring, 16) || !aligned(v_ring, 16) || !aligned(k_new, 16) || !aligned(v_new, 16) ||
      !aligned(lens, 4) || !aligned(depth, 4) || (err != nullptr && !aligned(err, 4)))
    return WMTP_EINVAL;
  wmtp::TreeAppendLaunch L{};
  L.k = static_cast<uint16_t*>(k_ring);
  L.v = static_cast<uint16_t*>(v_ring);
  L.k2 = static_cast<uint16_t*>(k_branch);
  L.v2 = static_cast<uint16_t*>(v_branch);
  L.k_new = static_cast<const uint16_t*>(k_new);
  L.v_new = static_cast<const uint16_t*>(v_new);
  L.lens = lens;
  L.depth = depth;
  L.err = err;
  L.B = B;
  L.width = width;
  L.Hkv = Hkv;
  L.d = d;
  L.sink = sink;
  L.R_w = R_w;
  L.dd = depth_max;
  if (wmtp::launch_tree_append(L, stream) != hipSuccess) return WMTP_ELAUNCH;
  return WMTP_OK;
}

WMTP_EXPORT int wmtp_tree_reset(int32_t* depth, int B, hipStream_t stream) {
  if (B < 0) return WMTP_EINVAL;
  if (B == 0) return WMTP_OK;
  if (depth == nullptr || !aligned(depth, 4)) return WMTP_EINVAL;
  if (wmtp::launch_rollback(depth, nullptr, B, nullptr, stream) != hipSuccess)
    return WMTP_ELAUNCH;
  return WMTP_OK;
}

WMTP_EXPORT int wmtp_ring_rollback(int32_t* lens, const int32_t* n_drop, int B, int32_t* err,
                                   hipStream_t stream) {
  if (B < 0) return WMTP_EINVAL;
  if (B == 0) return WMTP_OK;
  if (lens == nullptr || n_drop == nullptr || !aligned(lens, 4) || !aligned(n_drop, 4) ||
      (err != nullptr && !aligned(err, 4)))
    return WMTP_EINVAL;
  if (wmtp::launch_rollback(lens, n_drop, B, err, stream) != hipSuccess)
    return WMTP_ELAUNCH;
  return WMTP_OK;
}

WMTP_EXPORT int wmtp_fp8_quantize(const void* x, int64_t n, float scale, void* codes, hipStream_t stream) {
  if (n < 0 || n % 8 != 0 || !valid_scale(scale)) return WMTP_EINVAL;
  if (n == 0) return WMTP_OK;
  if (x == nullptr || codes == nullptr || !aligned(x, 16) || !aligned(codes, 8)) return WMTP_EINVAL;
  if (wmtp::launch_fp8_quantize(static_cast<const uint16_t*>(x), n, scale,
                                static_cast<uint8_t*>(codes),
                                stream) != hipSuccess)
    return WMTP_ELAUNCH;
  return WMTP_OK;
}

WMTP_EXPORT int wmtp_fp8_dequantize(const void* codes, int64_t n, void* out, hipStream_t stream) {
  if (n < 0 || n % 8 != 0) return WMTP_EINVAL;
  if (n == 0) return WMTP_OK;
  if (codes == nullptr || out == nullptr || !aligned(codes, 8) || !aligned(out, 16)) return WMTP_EINVAL;
  if (wmtp::launch_fp8_dequantize(static_cast<const uint8_t*>(codes), n, static_cast<uint16_t*>(out),
                                  stream) != hipSuccess)
    return WMTP_ELAUNCH;
  return WMTP_OK;
}

WMTP_EXPORT int wmtp_select_indices(const int32_t* lens, int B, int W, int sink, int R_w,
                                    int32_t* pos_out, int32_t* slot_out, int32_t* n_sel_out,
                                    int32_t* err, hipStream_t stream) {
  if (B < 0 || check_window(W, sink) != WMTP_OK) return WMTP_EINVAL;
  if (slot_out != nullptr && R_w < W) return WMTP_EINVAL;
  if (B == 0) return WMTP_OK;
  if (lens == nullptr || pos_out == nullptr || n_sel_out == nullptr) return WMTP_EINVAL;
  if (!aligned(lens, 4) || !aligned(pos_out, 4) || !aligned(n_sel_out, 4) ||
      (slot_out != nullptr && !aligned(slot_out, 4)) || (err != nullptr && !aligned(err, 4)))
    return WMTP_EINVAL;
  if (wmtp::launch_select(lens, B, W, sink, slot_out != nullptr ? R_w : W, pos_out, slot_out,
                          n_sel_out, err, stream) != hipSuccess)
    return WMTP_ELAUNCH;
  return WMTP_OK;
}

WMTP_EXPORT int wmtp_hbm_read_probe(const void* buf, int64_t bytes, uint32_t* sink, hipStream_t stream) {
  if (bytes < 0 || bytes % 16 != 0) return WMTP_EINVAL;
  if (bytes == 0) return WMTP_OK;
  if (buf == nullptr || sink == nullptr || !aligned(buf, 16) || !aligned(sink, 4)) return WMTP_EINVAL;
  if (wmtp::launch_hbm_read(buf, bytes, sink, stream) != hipSuccess)
    return WMTP_ELAUNCH;
  return WMTP_OK;
}

// ---------------------------------------------------------------------------
// Allocation-free windowed attention: the split partials live in a static
// device array (one copy per GPU, loaded with the library's code object and
// kept until the process ends) instead of a caller workspace.
//
// In host code `scratch` names a host-side stand-in, not device memory: its
// device address is resolved once per device with hipGetSymbolAddress and
// only that address is ever passed to a kernel.
static __device__ __align__(256) unsigned char scratch[WMTP_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int kScratchDevices = 64;
std::atomic<void*> g_scratch_ptr[kScratchDevices];
std::mutex g_scratch_mu;

// Device address of the current device's copy of `scratch`, resolved on the
// first call on that device (no allocation: the array is part of the code
// object).  Returns WMTP_ELAUNCH when the runtime cannot resolve it.
int scratch_address(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kScratchDevices) {
    (void)hipGetLastError();
    return WMTP_ELAUNCH;
  }
  void* p = g_scratch_ptr[dev].load(std::memory_order_acquire);
  if (p == nullptr) {
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    p = g_scratch_ptr[dev].load(std::memory_order_relaxed);
    if (p == nullptr) {
      void* addr = nullptr;
      if (hipGetSymbolAddress(&addr, HIP_SYMBOL(scratch)) != hipSuccess || addr == nullptr) {
        (void)hipGetLastError();
        return WMTP_ELAUNCH;
      }
      p = addr;
      g_scratch_ptr[dev].store(p, std::memory_order_release);
    }
  }
  *out = p;
  return WMTP_OK;
}

}  // namespace

WMTP_EXPORT int wmtp_draft_attn_windowed_noalloc(const void* q, const void* k, const void* v,
                                                 const int32_t* lens, void* out, float* lse, int B,
                                                 int Hq, int Hkv, int d, int64_t S_max, int W,
                                                 int sink, float scale, int32_t* err,
                                                 hipStream_t stream) {
  // Every argument check of the workspace form first (nothing enqueued),
  // then the partials of this shape against the static array.
  int st = attention_common(WMTP_VARIANT_WINDOWED, q, k, v, lens, nullptr, 1, out, lse, B, Hq, Hkv,
                            d, S_max, W, sink, W, scale, nullptr, 0, err, stream, nullptr, 0, false,
                            1.0f, 1.0f, nullptr, nullptr, 0, false, nullptr, true, false);
  if (st != WMTP_OK || B == 0) return st;
  const size_t need = wmtp_workspace_bytes(B, Hq, Hkv, d, S_max, W, sink, WMTP_VARIANT_WINDOWED);
  if (need > WMTP_NOALLOC_SCRATCH_BYTES) return WMTP_ESCRATCH;
  void* ptr = nullptr;
  st = scratch_address(&ptr);
  if (st != WMTP_OK) return st;
  return attention_common(WMTP_VARIANT_WINDOWED, q, k, v, lens, nullptr, 1, out, lse, B, Hq, Hkv,
                          d, S_max, W, sink, W, scale, ptr, WMTP_NOALLOC_SCRATCH_BYTES, err, stream);
}

WMTP_EXPORT const char* wmtp_status_string(int status) {
  switch (status) {
    case WMTP_OK: return "WMTP_OK";
    case WMTP_EINVAL: return "WMTP_EINVAL: invalid argument";
    case WMTP_EUNSUPPORTED: return "WMTP_EUNSUPPORTED: shape without a built kernel";
    case WMTP_EWORKSPACE: return "WMTP_EWORKSPACE: workspace too small";
    case WMTP_ELAUNCH: return "WMTP_ELAUNCH: kernel launch failed";
    case WMTP_ESCRATCH:
      return "WMTP_ESCRATCH: the call needs more scratch than the static array holds "
             "(WMTP_NOALLOC_SCRATCH_BYTES); use the workspace form of the call";
    default: return "unknown wmtp status";
  }
}

WMTP_EXPORT int wmtp_abi_version(void) { return WMTP_ABI_VERSION; }
