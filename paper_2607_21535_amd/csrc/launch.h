// Internal launch interface between the C-ABI layer and the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace wmtp {

// One attention call, already validated on the host.
struct AttnLaunch {
  int variant;  // wmtp_variant
  bool kv_fp8;  // K/V are E4M3 codes (dense or ring variants) instead of bf16
  const uint16_t* q;
  const void* k;
  const void* v;
  const int32_t* lens;
  const int32_t* n_q;  // new query rows per sequence, or NULL (all qps rows)
  int qps;             // query rows per sequence (1 for a draft decode step)
  const int32_t* table;   // paged variants: req_to_token [B, table_stride]
  int64_t table_stride;
  uint16_t* out;
  float* lse;
  int32_t* err;
  int B, Hq, Hkv, d;
  int64_t rows;     // rows per sequence: S_max (dense), sink + R_w (ring); pool rows (paged)
  int64_t len_cap;  // largest valid lens[b]
  int W, sink, R_w;
  float scale;
  float k_scale, v_scale;  // per-tensor scales of an fp8 cache (1 for bf16)
  // Tree variant: n_q is the speculative depth per request; candidates
  // b >= 1 read their private runs from k2 / v2 [B, rows2, Hkv, d]
  const void* k2;
  const void* v2;
  int64_t rows2;
  int dd;  // largest speculative depth (private-run length)
  // Fused draft step (variants windowed / ring): n_q holds n_new, k2 /
  // v2 the new rows [B, dd = n_max, Hkv, d]; the split kernel writes them into
  // the cache and the merge writes lens_out = old length + rows appended.
  bool step;
  int32_t* lens_out;
  // split plan (from plan_split; full-context variants)
  bool per_seq;   // items sized from each sequence's last row (full-context extend)
  int target;     // work items per KV head to aim for
  int chunk_cap;  // largest work item, in keys
  int max_items;  // work items per KV head, upper bound over all lengths
  // windowed plan (from plan_window; every windowed variant)
  int win_keys;    // selected keys per work item
  int win_items;   // work items per query row and KV head
  int win_slices;  // value slices per work item (1, or d / kWinSlice)
  int32_t* tickets;
  float* pm;
  float* pl;
  float* pz;
  float* po;
};

// Every workspace starts with the ticket counters of the one-launch kernels
// (int32, zero between calls); the partial results of any call follow them,
// so calls of different variants and shapes can share one workspace without
// touching each other's counters.
constexpr size_t kTicketBytes = size_t(1) << 20;
constexpr int64_t kMaxTickets = static_cast<int64_t>(kTicketBytes / sizeof(int32_t));

struct SplitPlan {
  int target;      // work items per KV head to aim for
  int chunk_cap;   // largest work item, in keys (multiple of kChunkQuantum)
  int max_items;   // most work items per KV head for any lengths
  size_t bytes;    // workspace bytes
  size_t off_pm;   // byte offsets of the partial arrays inside the workspace
  size_t off_pl;
  size_t off_pz;
  size_t off_po;
};

// Split plan for a validated shape; B counts query rows (sequences x rows per
// sequence); n_keys_max = most keys one query row attends.  qps > 1: the plan
// of a full-context extend whose items are sized per sequence (qps rows per
// sequence), with room for up to qps times more partials.
SplitPlan plan_split(int variant, int B, int Hq, int Hkv, int d, int64_t n_keys_max, int qps = 1);

// Windowed calls run in one launch (window_attn.hip): fixed work items of
// `item_keys` selected keys per query row and KV head, the value columns cut
// into `slices` slices of kWinSlice (or whole rows), and the merge done by
// the workgroup that takes the last ticket of its (row, KV head, slice).
constexpr int kWinSlice = 64;          // value columns per slice when sliced
constexpr int kWinOneLaunchRows = 4;   // query rows x KV heads up to which the one-launch kernel runs
constexpr int kWinMaxItemKeys = 1024;  // largest item (a paged item's pool rows live in LDS)
constexpr int64_t kWinFullMaxKeys = 16384;  // full-context capacity up to which the one-launch kernel runs (d = 256; a quarter below)

struct WinPlan {
  int item_keys;  // selected keys per work item (multiple of kChunkQuantum)
  int n_items;    // work items per query row and KV head (0: the shape needs
                  // more than kMaxTickets counters)
  int slices;     // value slices
  size_t bytes;   // workspace bytes (tickets + partials)
  size_t off_pm;  // byte offsets inside the workspace (tickets at 0)
  size_t off_pl;
  size_t off_pz;
  size_t off_po;
};

// Plan of a windowed call: NV query rows, at most `keys` = sink + W selected
// keys per row.  Depends only on the shape (not on lengths, cache capacity or
// the cache's element type), so the dense, ring and paged forms of one shape
// split identically and give bit-identical results.
WinPlan plan_window(int NV, int Hq, int Hkv, int d, int keys);

// Whether a windowed call of NV query rows runs the one-launch kernel (few
// rows: latency-bound single decodes) or the split-K kernel plus the merge
// kernel (many rows: the merge is spread over one workgroup per row and
// head).  Depends only on the shape, like the plans.
bool use_window_kernel(int NV, int Hkv);

// The multi-row extend kernel addresses a 64-key step with 32-bit byte
// offsets from the step's first token row (all KV heads): 64 rows must span
// less than 4 GiB.  Larger shapes take the per-row split kernel.
inline bool rows_kernel_fits(int Hkv, int d, bool fp8) {
  return 64LL * Hkv * d * (fp8 ? 1 : 2) < (1LL << 32);
}
bool use_window_kernel_full(int NV, int Hkv, int d, int64_t S_max);

hipError_t launch_window(const AttnLaunch& a, hipStream_t stream);

// Compute units of the current device (cached per device).
int device_cus();

// Index builder: kv_indptr [B+1] and kv_indices (packed) of the kept keys,
// each entry req_to_token[b][position] (variant: full or windowed key set).
hipError_t launch_kv_indices(const int32_t* table, int64_t table_stride, const int32_t* lens,
                             int B, bool windowed, int W, int sink, int64_t n_keys_max,
                             int32_t* indptr, int32_t* indices, int32_t* err, hipStream_t stream);

hipError_t launch_attention(const AttnLaunch& a, hipStream_t stream);

struct AppendLaunch {
  bool ring;
  bool fp8;  // quantise the bf16 rows to E4M3 codes (k_scale, v_scale)
  void* k;
  void* v;
  const uint16_t* k_new;
  const uint16_t* v_new;
  const int32_t* n_new;
  int32_t* lens;
  int32_t* err;
  int B, Hkv, d;
  int64_t rows;     // dense: S_max; ring: sink + R_w
  int sink, R_w, n_max;
  float k_scale, v_scale;
  int32_t* lens_out;  // NULL: lens is advanced in place; else lens is only read
};

hipError_t launch_append(const AppendLaunch& a, hipStream_t stream);

// Speculation bookkeeping.  Tree append: one draft row per candidate at
// position lens[b] + depth[b] (candidate 0 at its ring slot, candidate
// c >= 1 in its private run), then depth[b] += 1.
struct TreeAppendLaunch {
  uint16_t* k;  // ring [B, sink + R_w, Hkv, d]
  uint16_t* v;
  uint16_t* k2;  // private runs [B, (width - 1) * dd, Hkv, d]
  uint16_t* v2;
  const uint16_t* k_new;  // [B, width, Hkv, d]
  const uint16_t* v_new;
  const int32_t* lens;
  int32_t* depth;
  int32_t* err;
  int B, width, Hkv, d, sink, R_w, dd;
};
hipError_t launch_tree_append(const TreeAppendLaunch& a, hipStream_t stream);

// counts[b] -= n_drop[b] (n_drop NULL: counts[b] = 0), clamped at 0 and flagged.
hipError_t launch_rollback(int32_t* counts, const int32_t* n_drop, int B, int32_t* err, hipStream_t stream);

// Elementwise conversions of the fp8 cache format (the appends' quantiser and
// the attention's widening), n a multiple of 8.
hipError_t launch_fp8_quantize(const uint16_t* x, int64_t n, float scale, uint8_t* codes,
                               hipStream_t stream);
hipError_t launch_fp8_dequantize(const uint8_t* codes, int64_t n, uint16_t* out, hipStream_t stream);

// Streaming-read probe: WMTP_PROBE_BLOCKS workgroups read `bytes` (a multiple
// of 16) and each writes the XOR of its words to sink[block].
hipError_t launch_hbm_read(const void* buf, int64_t bytes, uint32_t* sink, hipStream_t stream);

hipError_t launch_select(const int32_t* lens, int B, int W, int sink, int R_w, int32_t* pos_out,
                         int32_t* slot_out, int32_t* n_sel_out, int32_t* err, hipStream_t stream);

}  // namespace wmtp
