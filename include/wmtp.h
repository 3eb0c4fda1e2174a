/*
 * wmtp.h -- C ABI of the Windowed-MTP draft decode attention library
 * (libwmtp.so, AMD Instinct MI355X / gfx950).
 *
 * The library computes the MTP draft head's single-token GQA decode attention
 * over its KV cache, as described in "Windowed-MTP: Removing the Full-Context
 * Draft-KV Tax at Million-Token Context":
 *   - full-context: the native draft attends every cached key (Section 3,
 *     per-step latency model; Figure "window", native row);
 *   - windowed: the draft attends the first `sink` keys plus the most recent
 *     `W` keys, and all keys while S <= sink + W (Section 4 "Mechanism";
 *     Appendix A, pseudocode of the windowing change);
 *   - ring: the same windowed attention over a compact per-request ring that
 *     stores only the sink and a circular window region (Section 4 and
 *     Section 6 "Memory"; the ring comment of the Appendix A pseudocode).
 *
 * Common conventions
 *   - All tensor pointers are DEVICE pointers owned by the caller.  The
 *     library allocates nothing, keeps no state between calls, never
 *     synchronises and only enqueues work on `stream` (a hipStream_t; NULL is
 *     the default stream).  Calls are safe to capture in a HIP graph.
 *   - bf16 tensors are raw bfloat16 bit patterns (uint16), row-major, and must
 *     be 16-byte aligned; int32 arrays must be 4-byte aligned.
 *   - Shapes: q and out [B, Hq, d]; a dense cache [B, S_max, Hkv, d]; a ring
 *     [B, sink + R_w, Hkv, d]; lens [B].  Query head h reads KV head
 *     h / (Hq / Hkv) (consecutive GQA grouping).
 *   - d must be 64, 128 or 256 and G = Hq / Hkv at most 16, otherwise
 *     WMTP_EUNSUPPORTED.  Other invalid arguments give WMTP_EINVAL; both are
 *     detected on the host before anything is enqueued.
 *   - Lengths live on the device (so a captured graph can replay a growing
 *     sequence).  lens[b] is the number of cached keys of sequence b, counting
 *     the current draft token's row.  A length outside its valid range is
 *     clamped on the device and WMTP_DERR_* bits are OR-ed into *err when
 *     `err` is not NULL.
 *   - Arithmetic: bf16 inputs, fp32 logits, softmax and accumulation; the
 *     softmax weights enter the weight-times-value product rounded to bf16
 *     and the output is normalised by the sum of those rounded weights; bf16
 *     output rounded to nearest even; lse (optional) is the natural-log
 *     log-sum-exp of the scaled logits from the fp32 weights.  An empty sequence (no keys)
 *     gives out = 0 and lse = -inf.
 *   - Results are deterministic: no atomics take part in any reduction.
 */
#ifndef WMTP_H
#define WMTP_H

#include <stddef.h>
#include <stdint.h>

/* The HIP stream handle: the same declaration as the HIP runtime header's,
 * so this header is usable with or without it (C11 and C++ accept the
 * repeated typedef).  NULL is the default stream. */
typedef struct ihipStream_t* hipStream_t;

#ifdef __cplusplus
extern "C" {
#endif

/* Host-side status codes. */
typedef enum {
  WMTP_OK = 0,
  WMTP_EINVAL = 1,        /* bad argument (null pointer, misalignment, bad size) */
  WMTP_EUNSUPPORTED = 2,  /* head size or GQA group outside the built kernels */
  WMTP_EWORKSPACE = 3,    /* ws_bytes smaller than wmtp_workspace_bytes() */
  WMTP_ELAUNCH = 4,       /* the HIP runtime rejected a kernel launch */
  WMTP_ESCRATCH = 5       /* the allocation-free call needs more than its static scratch */
} wmtp_status;

/* Device error bits, OR-ed into *err by the kernels. */
#define WMTP_DERR_LEN_RANGE 0x1  /* lens[b] < 0, > S_max for a dense cache, or < n_q[b]: clamped */
#define WMTP_DERR_NNEW_RANGE 0x2 /* n_new[b] outside [0, n_max] (n_q[b] outside [0, q_max]): clamped */
#define WMTP_DERR_CAPACITY 0x4   /* dense-cache append past S_max: extra rows dropped */
#define WMTP_DERR_SLOT_RANGE 0x8 /* req_to_token entry outside the pool: row 0 read instead */
#define WMTP_DERR_DEPTH 0x10     /* tree append at the largest speculative depth: nothing written */

/* Attention variants, for wmtp_workspace_bytes(). */
typedef enum {
  WMTP_VARIANT_FULL = 0,
  WMTP_VARIANT_WINDOWED = 1,
  WMTP_VARIANT_RING = 2,
  WMTP_VARIANT_PAGED_FULL = 3,
  WMTP_VARIANT_PAGED_WINDOWED = 4,
  WMTP_VARIANT_TREE = 5
} wmtp_variant;

/*
 * Workspace (device bytes) that one attention call of the given variant and
 * shape needs for its split-K partial results (per work item and query head:
 * the running maximum, two softmax denominators and the unnormalised output
 * row, in fp32) and its work counters, sized for the current device.  Small
 * calls (at most four query rows x KV heads; windowed, or full context over
 * at most 16384 cached rows per sequence at d = 256, 4096 below) run as one
 * launch whose last work item per row merges the others; their workspace
 * holds those items' records instead.
 * B counts query rows: the batch for the single-row calls, B * q_max for the
 * extend calls.  S_max is the dense cache capacity (ignored for the ring); W
 * and sink are ignored for the full variant.  Returns 0 for arguments the
 * attention calls would reject.
 * A workspace must be zero-filled once before its first use (for example
 * with hipMemset when it is allocated); every call leaves it ready for the
 * next call, so one workspace serves successive calls on one stream, also
 * replays of a captured graph.  Calls that may overlap in time need
 * separate workspaces.
 */
size_t wmtp_workspace_bytes(int B, int Hq, int Hkv, int d, int64_t S_max, int W, int sink,
                            int variant);

/*
 * Full-context draft decode attention (the native MTP draft; Section 3 and
 * the Figure "window" native row): every query token attends all keys
 * [0, lens[b]) of its sequence.
 *   q      [B, Hq, d] bf16           one draft query token per sequence
 *   k, v   [B, S_max, Hkv, d] bf16   dense draft KV cache, rows in position order
 *   lens   [B] int32 device          0 <= lens[b] <= S_max
 *   out    [B, Hq, d] bf16           attention output
 *   lse    [B, Hq] fp32 or NULL      natural-log log-sum-exp of the logits
 *   scale  logit scale (usually 1/sqrt(d)); must be finite
 *   ws, ws_bytes  workspace, see wmtp_workspace_bytes(..., WMTP_VARIANT_FULL)
 *   err    device int32 error word or NULL
 */
int wmtp_draft_attn_full(const void* q, const void* k, const void* v, const int32_t* lens,
                         void* out, float* lse, int B, int Hq, int Hkv, int d, int64_t S_max,
                         float scale, void* ws, size_t ws_bytes, int32_t* err, hipStream_t stream);

/*
 * Windowed draft decode attention over the dense cache (Section 4
 * "Mechanism"; Appendix A pseudocode): with S = lens[b], the kept keys are
 * [0, sink) and [S - W, S) when S > sink + W, and [0, S) otherwise -- at most
 * sink + W keys, whatever S is.  No other mask is applied.  Arguments as for
 * wmtp_draft_attn_full, plus
 *   W     recent-window length, >= 1 (the current token is always attended)
 *   sink  number of attention-sink keys, >= 0
 * Workspace: wmtp_workspace_bytes(..., WMTP_VARIANT_WINDOWED).
 */
int wmtp_draft_attn_windowed(const void* q, const void* k, const void* v, const int32_t* lens,
                             void* out, float* lse, int B, int Hq, int Hkv, int d, int64_t S_max,
                             int W, int sink, float scale, void* ws, size_t ws_bytes,
                             int32_t* err, hipStream_t stream);

/*
 * Allocation-free windowed draft decode attention, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation).  Computes exactly what
 * wmtp_draft_attn_windowed computes, with the same kernels, bit for bit, but
 * keeps the split partials in a static device array of
 * WMTP_NOALLOC_SCRATCH_BYTES inside the library (one per GPU, part of the
 * library's code object, held until the process ends) instead of a caller
 * workspace; the caller still passes inputs and outputs.  The call allocates
 * nothing and calls no allocating routine; its first call on a device
 * resolves the array's device address once.
 *   Returns WMTP_ESCRATCH (nothing enqueued) when the shape needs more
 *   partials than the array holds (wmtp_workspace_bytes of the windowed
 *   variant > WMTP_NOALLOC_SCRATCH_BYTES); other arguments and errors as for
 *   wmtp_draft_attn_windowed.
 *   Every call on one GPU uses that GPU's single array: calls that may
 *   overlap in time on one GPU (different streams, concurrent host threads)
 *   race on it and must be serialised by the caller.  Calls enqueued on one
 *   stream are ordered and safe.
 */
#define WMTP_NOALLOC_SCRATCH_BYTES (16u << 20)
int wmtp_draft_attn_windowed_noalloc(const void* q, const void* k, const void* v,
                                     const int32_t* lens, void* out, float* lse, int B, int Hq,
                                     int Hkv, int d, int64_t S_max, int W, int sink, float scale,
                                     int32_t* err, hipStream_t stream);

/*
 * Windowed draft decode attention over the compact ring store (Section 4 and
 * Section 6 "Memory": the draft KV pool shrinks to a fixed sink + window +
 * headroom footprint per request).  Logical position p of sequence b lives
 * in slot
 *     p                          if p < sink
 *     sink + ((p - sink) % R_w)  otherwise
 * of k_ring/v_ring [B, sink + R_w, Hkv, d]; lens[b] is the logical length
 * (any value >= 0).  R_w >= W keeps the whole window resident; the paper's
 * chain setting is R_w = W + gamma + 1 so rows of rejected draft tokens
 * never overwrite the live window.  The kept keys and their order are those
 * of wmtp_draft_attn_windowed, so the two calls give bit-identical outputs
 * for the same logical content.
 * Workspace: wmtp_workspace_bytes(..., WMTP_VARIANT_RING).
 */
int wmtp_ring_attn(const void* q, const void* k_ring, const void* v_ring, const int32_t* lens,
                   void* out, float* lse, int B, int Hq, int Hkv, int d, int W, int sink, int R_w,
                   float scale, void* ws, size_t ws_bytes, int32_t* err, hipStream_t stream);

/*
 * Draft-extend attention: several new query rows per sequence, attending
 * causally (the draft forward over the accepted tokens after a verify step;
 * "draft-extend attn" in the kernel attribution table, Appendix B, and the
 * discussion of ragged extend in Section 6 "The backend is not the confound").
 *   q, out  [B, q_max, Hq, d] bf16;  lse [B, q_max, Hq] fp32 or NULL
 *   lens    [B] int32 device: cached rows of sequence b INCLUDING its new rows
 *   n_q     [B] int32 device, 1..q_max: new rows of sequence b (NULL: q_max)
 * Row t < n_q[b] of sequence b attends the first lens[b] - n_q[b] + t + 1
 * cached rows -- the full context, or under the window rule applied at that
 * length (its own sink + last W); rows t >= n_q[b] give out = 0 and
 * lse = -inf.  A draft decode step is the case q_max = 1.  The ring variant
 * needs R_w >= W + q_max - 1 so that the earliest row's window is resident
 * (the paper's chain sizing R_w = W + gamma + 1 covers q_max = gamma + 1).
 * Workspace: at least wmtp_workspace_bytes(B * q_max, ..., variant).  Other
 * arguments and conventions as for the single-row calls.
 * The full-context form reads each sequence's keys once for all its rows,
 * cut into work items over the keys.  With only wmtp_workspace_bytes(B *
 * q_max, ...) bytes its items are sized from the keys of all rows, so a
 * sequence with n new rows spreads over about 1/n of the device's CUs; with
 * wmtp_extend_workspace_bytes(B, q_max, ...) bytes or more they are sized
 * from each sequence's last row (the one that sees every key) and fill the
 * device.  The two decompositions round differently; each is deterministic.
 */
size_t wmtp_extend_workspace_bytes(int B, int q_max, int Hq, int Hkv, int d, int64_t S_max, int W,
                                   int sink, int variant);
int wmtp_draft_extend_full(const void* q, const void* k, const void* v, const int32_t* lens,
                           const int32_t* n_q, void* out, float* lse, int B, int q_max, int Hq,
                           int Hkv, int d, int64_t S_max, float scale, void* ws, size_t ws_bytes,
                           int32_t* err, hipStream_t stream);
int wmtp_draft_extend_windowed(const void* q, const void* k, const void* v, const int32_t* lens,
                               const int32_t* n_q, void* out, float* lse, int B, int q_max, int Hq,
                               int Hkv, int d, int64_t S_max, int W, int sink, float scale,
                               void* ws, size_t ws_bytes, int32_t* err, hipStream_t stream);
int wmtp_ring_extend(const void* q, const void* k_ring, const void* v_ring, const int32_t* lens,
                     const int32_t* n_q, void* out, float* lse, int B, int q_max, int Hq, int Hkv,
                     int d, int W, int sink, int R_w, float scale, void* ws, size_t ws_bytes,
                     int32_t* err, hipStream_t stream);

/*
 * Paged draft KV (a shared token pool with page size 1, as in the paper's
 * serving setup, Section 4 "Mechanism" and Appendix A).  k_pool, v_pool
 * [pool_rows, Hkv, d] bf16 hold every request's rows; req_to_token
 * [B, table_stride] int32 gives the pool row of position p of request b
 * (0 <= lens[b] <= table_stride).  The attention reads pool rows through the
 * table only at the kept positions -- all of [0, lens[b]) natively, the sink
 * and the last W windowed -- and gives the same result, bit for bit, as the
 * dense call over a cache holding the same rows.  Table entries outside
 * [0, pool_rows) read row 0 and raise WMTP_DERR_SLOT_RANGE.
 * Workspace: wmtp_workspace_bytes(B, Hq, Hkv, d, table_stride, W, sink,
 * WMTP_VARIANT_PAGED_FULL / _WINDOWED).
 */
int wmtp_paged_attn_full(const void* q, const void* k_pool, const void* v_pool,
                         const int32_t* req_to_token, const int32_t* lens, void* out, float* lse,
                         int B, int Hq, int Hkv, int d, int64_t pool_rows, int64_t table_stride,
                         float scale, void* ws, size_t ws_bytes, int32_t* err, hipStream_t stream);
int wmtp_paged_attn_windowed(const void* q, const void* k_pool, const void* v_pool,
                             const int32_t* req_to_token, const int32_t* lens, void* out,
                             float* lse, int B, int Hq, int Hkv, int d, int64_t pool_rows,
                             int64_t table_stride, int W, int sink, float scale, void* ws,
                             size_t ws_bytes, int32_t* err, hipStream_t stream);

/*
 * The draft's KV-index builder (the step Windowed-MTP modifies, Appendix A
 * pseudocode: kv_index = req_to_token[r, keep]).  Writes kv_indptr [B + 1]
 * (prefix sums of the kept counts) and kv_indices (packed pool rows of the
 * kept keys, request by request, ascending position) for variant
 * WMTP_VARIANT_PAGED_FULL (keep all lens[b] positions: O(S)) or
 * WMTP_VARIANT_PAGED_WINDOWED (sink + last W: O(sink + W)).  `capacity` is
 * the length of kv_indices and must be at least
 * wmtp_kv_indices_capacity(variant, B, table_stride, W, sink); B <= 65535.
 */
int64_t wmtp_kv_indices_capacity(int variant, int B, int64_t table_stride, int W, int sink);
int wmtp_build_kv_indices(const int32_t* req_to_token, const int32_t* lens, int B,
                          int64_t table_stride, int variant, int W, int sink, int32_t* kv_indptr,
                          int32_t* kv_indices, int64_t capacity, int32_t* err, hipStream_t stream);

/*
 * Append draft KV rows to the ring store (the draft forward writes the K/V
 * row of each draft token it processes; Section 3 "Per-step latency model").
 * For each sequence b, rows k_new[b, i], v_new[b, i] for i < n_new[b] take
 * logical positions lens[b] + i and are written to their ring slots; then
 * lens[b] += n_new[b] on the device.  When n_new[b] exceeds the ring, only
 * rows that stay resident are written (the sink and the last R_w positions),
 * which equals writing every row in order.
 *   k_new, v_new  [B, n_max, Hkv, d] bf16;  n_new [B] int32 device, 0..n_max
 * One call must not run concurrently with an attention call on the same ring.
 */
int wmtp_ring_append(void* k_ring, void* v_ring, const void* k_new, const void* v_new,
                     const int32_t* n_new, int32_t* lens, int B, int Hkv, int d, int sink, int R_w,
                     int n_max, int32_t* err, hipStream_t stream);

/*
 * Append draft KV rows to a dense cache [B, S_max, Hkv, d]: rows go to
 * positions lens[b] .. lens[b] + n_new[b] - 1, then lens[b] += n_new[b].
 * Rows past S_max are dropped, lens[b] is clamped to S_max and
 * WMTP_DERR_CAPACITY is raised.  Other arguments as for wmtp_ring_append.
 */
int wmtp_cache_append(void* k, void* v, const void* k_new, const void* v_new,
                      const int32_t* n_new, int32_t* lens, int B, int Hkv, int d, int64_t S_max,
                      int n_max, int32_t* err, hipStream_t stream);

/*
 * Export of the windowed key selection and ring slot map that the attention
 * kernels use (for tests and debugging).  For each b and virtual key index
 * j < sink + W: pos_out[b, j] is the logical position of the j-th kept key
 * (ascending), or -1 for j >= n_sel; slot_out[b, j] (may be NULL) its ring
 * slot for ring window R_w (-1 past n_sel); n_sel_out[b] = min(lens[b],
 * sink + W).  lens[b] < 0 is clamped to 0 and flagged.  R_w is only used for
 * slot_out and must then be >= W.
 */
int wmtp_select_indices(const int32_t* lens, int B, int W, int sink, int R_w, int32_t* pos_out,
                        int32_t* slot_out, int32_t* n_sel_out, int32_t* err, hipStream_t stream);

/*
 * Fused draft step: the append and the attention of one draft step in one
 * call (the draft forward writes its token's K/V row, then attends; Section
 * 3, per-step latency model).  For each sequence b, the n_new[b] rows
 * k_new[b, i], v_new[b, i] (i < n_new[b] <= n_max) take positions
 * lens_in[b] + i; the one query row q[b] attends at length
 * lens_in[b] + n_new[b] (full, windowed, or windowed over the ring), reading
 * the new rows from k_new / v_new; the rows are written into the cache
 * (ring: the resident ones) and lens_out[b] = lens_in[b] + n_new[b].
 * Results, cache contents and lengths equal those of wmtp_cache_append /
 * wmtp_ring_append followed by the attention call, bit for bit.  The
 * windowed and ring steps are one launch fewer (the attention reads the new
 * rows from k_new / v_new and writes them into the cache); the full step
 * runs the append and then the full attention (redirecting the new rows
 * would cost the O(S) kernel more than the launch it saves).  lens_in is
 * only read and lens_out only written; they must be
 * different arrays (a draft loop alternates two).  A dense cache that would
 * grow past S_max keeps the rows that fit, lens_out is clamped and
 * WMTP_DERR_CAPACITY raised.  k_new, v_new [B, n_max, Hkv, d] bf16 (may be
 * NULL when n_max == 0); workspace as for the attention call of the same
 * variant.  The ring needs R_w >= W.
 */
int wmtp_draft_step_full(const void* q, void* k, void* v, const void* k_new, const void* v_new,
                         const int32_t* n_new, const int32_t* lens_in, int32_t* lens_out,
                         void* out, float* lse, int B, int Hq, int Hkv, int d, int64_t S_max,
                         int n_max, float scale, void* ws, size_t ws_bytes, int32_t* err,
                         hipStream_t stream);
int wmtp_draft_step_windowed(const void* q, void* k, void* v, const void* k_new,
                             const void* v_new, const int32_t* n_new, const int32_t* lens_in,
                             int32_t* lens_out, void* out, float* lse, int B, int Hq, int Hkv,
                             int d, int64_t S_max, int n_max, int W, int sink, float scale,
                             void* ws, size_t ws_bytes, int32_t* err, hipStream_t stream);
int wmtp_ring_step(const void* q, void* k_ring, void* v_ring, const void* k_new,
                   const void* v_new, const int32_t* n_new, const int32_t* lens_in,
                   int32_t* lens_out, void* out, float* lse, int B, int Hq, int Hkv, int d, int W,
                   int sink, int R_w, int n_max, float scale, void* ws, size_t ws_bytes,
                   int32_t* err, hipStream_t stream);

/*
 * Speculative draft rows.
 *
 * Chain rollback: a chain that appends its speculative draft rows with
 * wmtp_ring_append (lens advancing with each) discards the rows the target
 * rejected by lowering lens: lens[b] -= n_drop[b] on the device (n_drop
 * outside [0, lens[b]] is clamped and flagged WMTP_DERR_NNEW_RANGE).  The
 * rows stay in their slots and are overwritten by later appends.  Every row
 * a later windowed read needs is still held when R_w >= W + (rows appended
 * past the committed length) -- the paper's chain ring of
 * n_sink + W + d slots (Section 7, tree speculation; Appendix A ring
 * comment).
 */
int wmtp_ring_rollback(int32_t* lens, const int32_t* n_drop, int B, int32_t* err, hipStream_t stream);

/*
 * Tree-width rings (Section 7, tree speculation).  Sizing rule: every
 * candidate of a tree reads the same sink and window rows; only its own most
 * recent d draft rows are private to it, so k candidates need the chain's
 * n_sink + W + d slots plus d more for each further candidate, d k in all.
 *   State per request: lens[b] = committed length S (rows the target has
 *   accepted), depth[b] = speculative depth i (0 .. depth_max), both on the
 *   device.  Candidate c's sequence is rows [0, S) followed by its own rows
 *   at positions S .. S + i - 1.
 *   Layout: the ring [B, sink + R_w, Hkv, d] with R_w >= W + depth_max holds
 *   the committed rows and candidate 0's rows at their ring slots (in place,
 *   as a chain writes them); the private runs [B, (width - 1) * depth_max,
 *   Hkv, d] hold candidate c >= 1's row of position S + t at run row
 *   (c - 1) * depth_max + t.  Sink + W + depth_max * width rows in all.
 *   k_branch / v_branch may be NULL when width == 1.
 * wmtp_tree_append: k_new, v_new [B, width, Hkv, d] bf16, one draft row per
 *   candidate, written for position S + depth[b]; then depth[b] += 1.  A
 *   request already at depth_max is left unchanged and flagged
 *   WMTP_DERR_DEPTH.
 * wmtp_tree_attn: q, out [B, width, Hq, d] bf16, lse [B, width, Hq] or NULL.
 *   Candidate c of request b attends the windowed key set (sink + W) of its
 *   own sequence at length S + depth[b].  Workspace:
 *   wmtp_workspace_bytes(B * width, Hq, Hkv, d, 0, W, sink, WMTP_VARIANT_TREE).
 * wmtp_tree_reset: depth[b] = 0 for every request (after the verify).  The
 *   accepted tokens' draft rows are then written at their committed
 *   positions by wmtp_ring_append + wmtp_ring_extend (the draft-extend step,
 *   at most depth_max + 1 rows, which the R_w >= W + depth_max headroom
 *   allows).
 */
int wmtp_tree_append(void* k_ring, void* v_ring, void* k_branch, void* v_branch, const void* k_new,
                     const void* v_new, const int32_t* lens, int32_t* depth, int B, int width,
                     int Hkv, int d, int W, int sink, int R_w, int depth_max, int32_t* err,
                     hipStream_t stream);
int wmtp_tree_attn(const void* q, const void* k_ring, const void* v_ring, const void* k_branch,
                   const void* v_branch, const int32_t* lens, const int32_t* depth, void* out,
                   float* lse, int B, int width, int Hq, int Hkv, int d, int W, int sink, int R_w,
                   int depth_max, float scale, void* ws, size_t ws_bytes, int32_t* err,
                   hipStream_t stream);
int wmtp_tree_reset(int32_t* depth, int B, hipStream_t stream);

/*
 * fp8 draft KV cache (Section 7, KV-cache quantization: the windowing
 * composes with fp8 KV; the dtype sets the bytes per entry, windowing the
 * number of entries read).  Format: OCP E4M3 ("e4m3fn": bias 7, subnormals,
 * no infinities, largest finite 448), one byte per element, with one float32
 * scale per tensor: code c of the key cache stands for value(c) * k_scale,
 * of the value cache for value(c) * v_scale.  Layouts are those of the bf16
 * cache with 1-byte elements ([B, S_max, Hkv, d] dense, [B, sink + R_w, Hkv,
 * d] ring), 16-byte aligned.  q, out and lse are as for the bf16 calls, and
 * so is the workspace (wmtp_workspace_bytes of the same variant).
 *
 * Attention: the same definition over the dequantized cache.  Codes are
 * widened to bf16 exactly (every E4M3 value is a bf16 value); k_scale is
 * folded into the logit scale, v_scale into the output normalisation.
 * k_scale and v_scale must be finite and positive (else WMTP_EINVAL).
 */
int wmtp_draft_attn_full_fp8(const void* q, const void* k, const void* v, const int32_t* lens,
                             void* out, float* lse, int B, int Hq, int Hkv, int d, int64_t S_max,
                             float scale, float k_scale, float v_scale, void* ws, size_t ws_bytes,
                             int32_t* err, hipStream_t stream);
int wmtp_draft_attn_windowed_fp8(const void* q, const void* k, const void* v, const int32_t* lens,
                                 void* out, float* lse, int B, int Hq, int Hkv, int d,
                                 int64_t S_max, int W, int sink, float scale, float k_scale,
                                 float v_scale, void* ws, size_t ws_bytes, int32_t* err,
                                 hipStream_t stream);
int wmtp_ring_attn_fp8(const void* q, const void* k_ring, const void* v_ring, const int32_t* lens,
                       void* out, float* lse, int B, int Hq, int Hkv, int d, int W, int sink,
                       int R_w, float scale, float k_scale, float v_scale, void* ws,
                       size_t ws_bytes, int32_t* err, hipStream_t stream);

/*
 * fp8 paged draft attention (Section 7 KV-cache quantization over the paged
 * pool of Section 4 / Appendix A): wmtp_paged_attn_full / _windowed over a
 * pool of E4M3 codes, k_pool and v_pool [pool_rows, Hkv, d] uint8 (16-byte
 * aligned), with the per-tensor scales of the fp8 cache calls.  Results
 * equal, bit for bit, the fp8 dense call over a cache holding the same rows.
 * Workspace and error bits as for the bf16 paged calls.
 */
/*
 * fp8 draft-extend: the draft-extend calls (several causal new rows per
 * sequence, as wmtp_draft_extend_full / _windowed / wmtp_ring_extend) over
 * an fp8 dense cache or ring, with the per-tensor scales of the fp8 calls.
 * The full-context form reads the context once for all new rows, as the
 * bf16 form (at d = 64, once per row).
 */
int wmtp_draft_extend_full_fp8(const void* q, const void* k, const void* v, const int32_t* lens,
                               const int32_t* n_q, void* out, float* lse, int B, int q_max,
                               int Hq, int Hkv, int d, int64_t S_max, float scale, float k_scale,
                               float v_scale, void* ws, size_t ws_bytes, int32_t* err,
                               hipStream_t stream);
int wmtp_draft_extend_windowed_fp8(const void* q, const void* k, const void* v,
                                   const int32_t* lens, const int32_t* n_q, void* out, float* lse,
                                   int B, int q_max, int Hq, int Hkv, int d, int64_t S_max, int W,
                                   int sink, float scale, float k_scale, float v_scale, void* ws,
                                   size_t ws_bytes, int32_t* err, hipStream_t stream);
int wmtp_ring_extend_fp8(const void* q, const void* k_ring, const void* v_ring,
                         const int32_t* lens, const int32_t* n_q, void* out, float* lse, int B,
                         int q_max, int Hq, int Hkv, int d, int W, int sink, int R_w, float scale,
                         float k_scale, float v_scale, void* ws, size_t ws_bytes, int32_t* err,
                         hipStream_t stream);

int wmtp_paged_attn_full_fp8(const void* q, const void* k_pool, const void* v_pool,
                             const int32_t* req_to_token, const int32_t* lens, void* out,
                             float* lse, int B, int Hq, int Hkv, int d, int64_t pool_rows,
                             int64_t table_stride, float scale, float k_scale, float v_scale,
                             void* ws, size_t ws_bytes, int32_t* err, hipStream_t stream);
int wmtp_paged_attn_windowed_fp8(const void* q, const void* k_pool, const void* v_pool,
                                 const int32_t* req_to_token, const int32_t* lens, void* out,
                                 float* lse, int B, int Hq, int Hkv, int d, int64_t pool_rows,
                                 int64_t table_stride, int W, int sink, float scale,
                                 float k_scale, float v_scale, void* ws, size_t ws_bytes,
                                 int32_t* err, hipStream_t stream);

/*
 * fp8 appends: as wmtp_ring_append / wmtp_cache_append, with the bf16 rows
 * quantised on the way in.  Element x of a key row is stored as the E4M3
 * code nearest to x / k_scale (division in float32, correctly rounded),
 * saturated to +-448, ties to the even code; values likewise with v_scale.
 * Non-finite inputs are outside the contract.
 */
int wmtp_ring_append_fp8(void* k_ring, void* v_ring, const void* k_new, const void* v_new,
                         const int32_t* n_new, int32_t* lens, int B, int Hkv, int d, int sink,
                         int R_w, int n_max, float k_scale, float v_scale, int32_t* err,
                         hipStream_t stream);
int wmtp_cache_append_fp8(void* k, void* v, const void* k_new, const void* v_new,
                          const int32_t* n_new, int32_t* lens, int B, int Hkv, int d,
                          int64_t S_max, int n_max, float k_scale, float v_scale, int32_t* err,
                          hipStream_t stream);

/*
 * The fp8 format's element conversions, as the appends and the attention
 * kernels perform them (for tests and for filling a cache in bulk):
 * quantize writes codes[i] for bf16 x[i] with `scale` (the appends' rule);
 * dequantize writes the bf16 value of codes[i] (exact; NaN codes give NaN).
 * n must be a multiple of 8; x and out 16-byte, codes 8-byte aligned.
 */
int wmtp_fp8_quantize(const void* x, int64_t n, float scale, void* codes, hipStream_t stream);
int wmtp_fp8_dequantize(const void* codes, int64_t n, void* out, hipStream_t stream);

/*
 * Measurement helper, not part of the method: one streaming pass over `bytes`
 * bytes of device memory at `buf` with the attention kernels' load type
 * (16-byte non-temporal loads), in WMTP_PROBE_BLOCKS workgroups.  Timed by
 * the caller, its rate is the device's practical HBM read ceiling.
 *   bytes   a multiple of 16 (0: nothing is launched); buf 16-byte aligned
 *   sink    uint32[WMTP_PROBE_BLOCKS] device: workgroup i writes the XOR of
 *           the 32-bit words it read, so the XOR over sink is the XOR of
 *           every word of the buffer
 * Returns WMTP_EINVAL for a bad size, pointer or alignment.
 */
#define WMTP_PROBE_BLOCKS 512
int wmtp_hbm_read_probe(const void* buf, int64_t bytes, uint32_t* sink, hipStream_t stream);

/* Human-readable name of a wmtp_status value (static string). */
const char* wmtp_status_string(int status);

/* ABI version of this header, (major << 16) | minor. */
int wmtp_abi_version(void);

#define WMTP_ABI_VERSION ((2 << 16) | 2)

#ifdef __cplusplus
}
#endif

#endif /* WMTP_H */
