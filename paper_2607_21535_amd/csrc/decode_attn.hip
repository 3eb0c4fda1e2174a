// Split-K GQA decode attention for gfx950 (full, windowed, ring, paged, tree
// and fused-step key maps; bf16 or fp8 cache), a multi-row variant for the
// full-context draft-extend, and the log-sum-exp merge of the split partials.
//
// What is computed: for every sequence b and query head h, softmax attention
// of q[b,h] over the keys the variant selects (Windowed-MTP Section 4
// "Mechanism" and the Appendix A pseudocode; the native draft reads all S
// keys, Section 3).  The selection is the O(1) index arithmetic of
// index_map.h; no index table is built.
//
// Work decomposition.  Sequence b attends n_sel(b) keys, cut into work items
// whose size the kernels derive on the device from the batch's total
// selected keys (so a captured graph adapts to the lengths of each replay);
// the items of all sequences are numbered consecutively (a prefix sum over
// the device-resident lengths, so variable-length batches pack without
// holes) and one 256-thread workgroup handles one (item, KV head).  The four
// waves of a workgroup take interleaved 16-key tiles, so the group streams
// one contiguous key range; each tile's K rows pass through LDS on their way
// to the MFMA (whole-row loads), its V values go straight to registers.
//
// Per 16-key tile, on one wave:
//   S^T[16 keys, 16 heads] = K_tile . Q^T   v_mfma_f32_16x16x32_bf16, d/32 steps
//   online softmax per head in the exp2 domain (scale * log2 e folded into the
//   fp32 logits); a head's 16 scores sit in four lanes (two xor shuffles)
//   O^T[d, heads] += V^T . P^T              v_mfma_f32_16x16x16_bf16, d/16 steps
// In this orientation a query head sits on the same lane in the scores and
// in the output accumulator (rescaling is lane-local), and each lane already
// holds, for every value column it loaded, the four keys its lane group
// contributes to the PV product: two byte permutes build the MFMA operand,
// with no transpose through LDS.  P is rounded to bf16 for that product; the
// output is normalised by the sum of the same rounded weights, and the
// log-sum-exp uses the fp32 weights.
// The four waves combine their state in a fixed order (m, l, z through LDS,
// O pairwise in registers), and the merge kernel combines the items of a
// sequence in a fixed order: results are bitwise reproducible.
//
// Query heads beyond G in the 16-wide MFMA operand are zero and discarded.

#include "../../include/wmtp.h"
#include "common.h"
#include "fp8.h"
#include "attn_device.h"
#include "index_map.h"
#include "launch.h"

#include <algorithm>
#include <atomic>
#include <climits>
#include <cstdlib>
#include <type_traits>

#ifndef WMTP_CHUNK_MAX_DEFAULT
#define WMTP_CHUNK_MAX_DEFAULT 9216
#endif

namespace wmtp {
namespace {

constexpr int kMergeThreads = 1024;
constexpr int kPagedChunkMax = 9216;  // largest work item of a paged call (its slots live in LDS)

struct SplitArgs {
  const uint16_t* q;
  const void* k;  // bf16 or fp8 elements
  const void* v;
  const int32_t* lens;
  float* pm;
  float* pl;
  float* pz;
  float* po;
  int32_t* err;
  const int32_t* n_q;  // new query rows per sequence (NULL: all qps rows)
  const int32_t* table;  // paged: req_to_token [B, table_stride]
  int64_t table_stride;
  int B, Hq, Hkv, G;
  int qps;             // query rows per sequence; NV = B * qps query rows in all
  int64_t rows;        // dense: rows per sequence; ring: slots; paged: pool rows
  int64_t len_cap;
  int W, sink, R_w;
  int target;     // work items per KV head to aim for
  int chunk_cap;  // largest item, in keys
  float scale_log2;
  // Tree: n_q holds each request's speculative depth (0 .. dd); candidate
  // b >= 1 reads its private run from k2 / v2 [B, rows2, Hkv, D]
  const void* k2;
  const void* v2;
  int64_t rows2;
  int dd;
  int per_seq;  // item size from each sequence's last row only (see wave_chunk)
};

struct MergeArgs {
  const int32_t* lens;
  const float* pm;
  const float* pl;
  const float* pz;
  const float* po;
  uint16_t* out;
  float* lse;
  int32_t* err;
  const int32_t* n_q;
  int B, Hq, Hkv, G;
  int qps;
  int64_t len_cap;
  int W, sink, target, chunk_cap;
  float out_scale;  // value scale of an fp8 cache (1 for bf16)
  int dd;           // Tree: largest speculative depth; fused step: n_max
  int32_t* lens_out;  // fused step: each row's new length
  int per_seq;        // as in SplitArgs
};

// Work decomposition, derived the same way by every split and merge
// workgroup from the device-resident lengths (so a captured graph adapts to
// the lengths of each replay): the item size is the batch's total number of
// selected keys per KV head divided by `target`, rounded up to a multiple of
// kChunkQuantum and clamped to [kChunkQuantum, chunk_cap]; sequence b owns
// ceil(n_sel(b) / chunk) consecutive items (per query row, see
// visible_len).  per_seq (full-context draft-extend with a workspace for
// it): the total counts only the last new row of each sequence, the one
// that sees every key, so the multi-row kernel, which reads a sequence's
// keys once for all its rows, gets about `target` items per KV head however
// many rows share them (each row still has its own partials).  Runs on one
// whole wave; every lane returns the same value.  `first` receives the
// visible length of row `lane` (0 past the last row), so that a scan over
// the first 64 rows need not read the lengths again.
template <KeyMap M>
__device__ int wave_chunk(const int32_t* lens, const int32_t* n_q, int qps, int NV, int64_t len_cap,
                          int W, int sink, int target, int chunk_cap, int32_t* err, bool report, int dd,
                          bool per_seq, int& first) {
  const int lane = threadIdx.x & (kWave - 1);
  long long total = 0;
  first = 0;
  for (int base = 0; base < NV; base += kWave) {
    const int v = base + lane;
    int b;
    if (v < NV) {
      const int S = visible_len<M>(lens, n_q, qps, len_cap, err, v, report, b, dd);
      if (base == 0) first = S;
      // per_seq: only the sequence's last new row (n = n_q[b], clamped as
      // in visible_len) counts; a select rather than a branch
      const int n = n_q == nullptr ? qps : min(max(n_q[b], 0), qps);
      const long long keys = selected_count<M>(S, W, sink);
      total += (!per_seq || v - b * qps == n - 1) ? keys : 0ll;
    }
  }
#pragma unroll
  for (int off = kWave / 2; off > 0; off >>= 1) total += __shfl_xor(total, off);
  long long c = (total + target - 1) / target;
  c = (c + kChunkQuantum - 1) / kChunkQuantum * kChunkQuantum;
  c = c < kChunkQuantum ? kChunkQuantum : (c > chunk_cap ? chunk_cap : c);
  return static_cast<int>(c);
}

// Finds the query row v and local chunk c of work item `item` (wave 0 scans
// the lengths; the result is broadcast through LDS).  Returns false for the
// whole workgroup when `item` lies past the last query row's items.
template <KeyMap M>
__device__ bool locate_item(const SplitArgs& a, int item, int& v_out, int& c_out, int& S_out,
                            int& chunk_out) {
  __shared__ int s_v, s_c, s_S, s_chunk;
  const int NV = a.B * a.qps;
  if (threadIdx.x < kWave) {
    const int lane = threadIdx.x;
    int first;
    const int chunk = wave_chunk<M>(a.lens, a.n_q, a.qps, NV, a.len_cap, a.W, a.sink, a.target,
                                    a.chunk_cap, a.err, true, a.dd, a.per_seq != 0, first);
    if (lane == 0) {
      s_v = -1;
      s_chunk = chunk;
    }
    int carry = 0;
    for (int base = 0; base < NV; base += kWave) {
      const int v = base + lane;
      int S = 0, cnt = 0;
      if (v < NV) {
        int b;
        S = base == 0 ? first : visible_len<M>(a.lens, a.n_q, a.qps, a.len_cap, a.err, v, false, b, a.dd);
        cnt = ceil_div_i(selected_count<M>(S, a.W, a.sink), chunk);
      }
      int incl = cnt;
#pragma unroll
      for (int off = 1; off < kWave; off <<= 1) {
        const int t = __shfl_up(incl, off);
        if (lane >= off) incl += t;
      }
      const int lo = carry + incl - cnt;
      if (cnt > 0 && item >= lo && item < lo + cnt) {
        s_v = v;
        s_c = item - lo;
        s_S = S;
      }
      carry += __shfl(incl, kWave - 1);
      if (carry > item) break;
    }
  }
  __syncthreads();
  v_out = s_v;
  c_out = s_c;
  S_out = s_S;
  chunk_out = s_chunk;
  return v_out >= 0;
}

// The kernel fits 256 registers per lane (two waves per SIMD at d = 256), so
// that two workgroups can share a CU when a call has more work items than
// the device has CUs (long batches); a single sequence takes one per CU.
template <int D, KeyMap M, bool F8>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2))) void split_kernel(SplitArgs a) {
  using KT = std::conditional_t<F8, uint8_t, uint16_t>;  // one cached K/V element
  constexpr int VEC = D / 16;  // d values of one key per lane in the PV operand
  // A lane's VEC values come in pieces of SEG contiguous d values (16 bytes at
  // most); piece s of lane col starts at d = s*16*SEG + SEG*col, so the 16
  // lanes of one key read 16*SEG contiguous values per load instruction.
  // fp8: one piece of VEC codes (at most 16 bytes).
  constexpr int SEG = F8 ? VEC : (VEC < 8 ? VEC : 8);
  constexpr int NSEG = VEC / SEG;
  constexpr int KCH = D / 32;  // 16x16x32 steps over d for the logits

  const int lane = threadIdx.x & (kWave - 1);
  // Wave-uniform values are moved to scalar registers so that the tile loop
  // is scalar control flow (exact load/wait accounting, no exec masking).
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const int grp = lane >> 4;  // 0..3
  const int col = lane & 15;  // query head (within the group) owned by this lane
  const int g = blockIdx.x % a.Hkv;
  const int item = blockIdx.x / a.Hkv;

  int v, c, S, chunk;
  if (!locate_item<M>(a, item, v, c, S, chunk)) return;
  v = __builtin_amdgcn_readfirstlane(v);
  const int b = a.qps == 1 ? v : v / a.qps;  // the sequence whose KV row v reads
  c = __builtin_amdgcn_readfirstlane(c);
  S = __builtin_amdgcn_readfirstlane(S);
  chunk = __builtin_amdgcn_readfirstlane(chunk);
  const int n_sel = selected_count<M>(S, a.W, a.sink);
  const int j0 = c * chunk;
  const int j1 = min(j0 + chunk, n_sel);
  RowMap<M> map(S, a.W, a.sink, a.R_w);
  if constexpr (has_tail(M)) {
    int s_commit;
    (void)tail_len<M>(a.lens, a.n_q, a.dd, a.len_cap, b, a.err, false, s_commit);
    map.S_c = s_commit;
    if constexpr (M == KeyMap::Tree) {
      const int cand = v - b * a.qps;
      map.bbase = cand == 0 ? -1 : static_cast<int>(a.rows) + (cand - 1) * a.dd;
    } else {
      map.bbase = static_cast<int>(a.rows);
    }
  }
  const int64_t rs = static_cast<int64_t>(a.Hkv) * D;  // elements between rows
  // Dense and ring caches hold `rows` rows per sequence; a paged pool is one
  // shared array of rows indexed by the request's token table.
  const int64_t seq_rows = is_paged(M) ? 0 : static_cast<int64_t>(b) * a.rows;
  const int64_t seq_off = (seq_rows * a.Hkv + g) * D;
  const KT* kbase = static_cast<const KT*>(a.k) + seq_off;
  const KT* vbase = static_cast<const KT*>(a.v) + seq_off;
  // Tree: rows at or past the ring's `rows` are in the candidate's private run.
  [[maybe_unused]] const int64_t off2 = (static_cast<int64_t>(b) * a.rows2 * a.Hkv + g) * D;
  auto key_row = [&](int r) -> const KT* {
    if constexpr (has_tail(M)) {
      if (r >= a.rows) return static_cast<const KT*>(a.k2) + off2 + static_cast<int64_t>(r - a.rows) * rs;
    }
    return kbase + static_cast<int64_t>(r) * rs;
  };
  auto value_row = [&](int r) -> const KT* {
    if constexpr (has_tail(M)) {
      if (r >= a.rows) return static_cast<const KT*>(a.v2) + off2 + static_cast<int64_t>(r - a.rows) * rs;
    }
    return vbase + static_cast<int64_t>(r) * rs;
  };

  // Fused draft step: the first work item of a row also writes its KV head's
  // slice of the appended rows into the cache (ring: the resident ones).  No
  // workgroup of this launch reads those slots: the appended positions are
  // read from the new-row buffer, and on a ring (R_w >= W) a slot they
  // overwrite held a position outside every window of this call.  A thread's
  // first unit is loaded here, beside the tile loads, and stored when the
  // workgroup is done (a store ahead of the tile loads would hold them up:
  // memory operations of a wave complete in order).
  [[maybe_unused]] constexpr int kCopyUnits = D / 8;  // 16-byte units per head row
  [[maybe_unused]] u32x4 cpy_k = {}, cpy_v = {};
  [[maybe_unused]] int64_t cpy_dst = -1;
  auto copy_unit = [&](int u, int64_t& src, int64_t& dst) -> bool {  // false: nothing to write for unit u
    const int i = u / kCopyUnits;
    const int off = (u % kCopyUnits) * 8;
    const int p = map.S_c + i;
    int slot = p;
    if constexpr (is_ring(M)) {
      if (p >= a.sink && p < S - a.R_w) return false;  // overwritten later in the same append
      slot = p < a.sink ? p : a.sink + (p - a.sink) % a.R_w;
    }
    src = off2 + static_cast<int64_t>(i) * rs + off;
    dst = static_cast<int64_t>(slot) * rs + off;
    return true;
  };
  if constexpr (is_step(M)) {
    int64_t src, dst;
    if (c == 0 && static_cast<int>(threadIdx.x) < (S - map.S_c) * kCopyUnits && copy_unit(threadIdx.x, src, dst)) {
      cpy_dst = dst;
      cpy_k = *reinterpret_cast<const u32x4*>(static_cast<const uint16_t*>(a.k2) + src);
      cpy_v = *reinterpret_cast<const u32x4*>(static_cast<const uint16_t*>(a.v2) + src);
    }
  }
  auto store_copy = [&]() {
    if constexpr (is_step(M)) {
      if (c == 0) {
        uint16_t* kw = const_cast<uint16_t*>(reinterpret_cast<const uint16_t*>(kbase));
        uint16_t* vw = const_cast<uint16_t*>(reinterpret_cast<const uint16_t*>(vbase));
        if (cpy_dst >= 0) {
          *reinterpret_cast<u32x4*>(kw + cpy_dst) = cpy_k;
          *reinterpret_cast<u32x4*>(vw + cpy_dst) = cpy_v;
        }
        for (int u = static_cast<int>(threadIdx.x) + kThreads; u < (S - map.S_c) * kCopyUnits; u += kThreads) {
          int64_t src, dst;  // long appends
          if (!copy_unit(u, src, dst)) continue;
          *reinterpret_cast<u32x4*>(kw + dst) = *reinterpret_cast<const u32x4*>(static_cast<const uint16_t*>(a.k2) + src);
          *reinterpret_cast<u32x4*>(vw + dst) = *reinterpret_cast<const u32x4*>(static_cast<const uint16_t*>(a.v2) + src);
        }
      }
    }
  };

  // Paged: the pool rows of this item's keys, looked up once into LDS.
  [[maybe_unused]] int* slots = nullptr;
  if constexpr (is_paged(M)) {
    __shared__ int s_slot[kPagedChunkMax];
    slots = s_slot;
    const int32_t* trow = a.table + static_cast<int64_t>(b) * a.table_stride;
    bool bad = false;
    for (int j = j0 + static_cast<int>(threadIdx.x); j < j1; j += kThreads) {
      int slot = trow[map.row(j)];
      if (slot < 0 || static_cast<int64_t>(slot) >= a.rows) {
        bad = true;
        slot = 0;
      }
      s_slot[j - j0] = slot;
    }
    if (bad) raise_error(a.err, WMTP_DERR_SLOT_RANGE);
    __syncthreads();
  }
  auto row_of = [&](int j) -> int {
    if constexpr (is_paged(M)) {
      return slots[j - j0];
    } else {
      return map.row(j);
    }
  };

  // Q^T operand: lane (grp, col) holds at step kk the 8 d values of head col
  // that the key operand holds: d = kk*32 + grp*8 (bf16 keys) or
  // (kk/2*4 + grp)*16 + (kk%2)*8 (fp8 keys: 16 codes per load).
  bf16x8 qf[KCH];
  {
    const bool live = col < a.G;
    const uint16_t* qp = a.q + (static_cast<int64_t>(v) * a.Hq + g * a.G + (live ? col : 0)) * D;
#pragma unroll
    for (int kk = 0; kk < KCH; ++kk) {
      const int d0 = F8 ? ((kk >> 1) * 4 + grp) * 16 + (kk & 1) * 8 : kk * 32 + grp * 8;
      u32x4 w = *reinterpret_cast<const u32x4*>(qp + d0);
      if (!live) w = u32x4{0u, 0u, 0u, 0u};
      qf[kk] = __builtin_bit_cast(bf16x8, w);
    }
  }

  using Tile = TileRegs<D, F8>;

  // Keys reach the MFMA through LDS: the tile's K rows are loaded key-major
  // and contiguous (16-byte units f = 64 i + lane), each wave stores them into
  // its own padded LDS tile and reads the operand back (lane (grp, col): key
  // col, unit 4 kk + grp; an fp8 unit holds 16 codes, two MFMA steps).  A load
  // instruction then covers whole 256..512-byte runs of two to eight keys
  // instead of 64-byte pieces of sixteen, which HBM serves about 10% faster.
  // The row pitch (two units of padding) makes the operand reads free of
  // bank conflicts (gfx950 LDS serves them at its full 256 bytes per clock;
  // one unit of padding halves that).  A wave's own stores
  // and loads are processed in order: no barrier is needed.  The epilogue
  // reuses the same LDS (after a barrier every wave has passed its last tile).
  constexpr int kKUnits = F8 ? D / 16 : D / 8;  // 16-byte units per key row (one KV head)
  constexpr int kKPitch = kKUnits + 2;          // LDS row pitch in units
  constexpr int kKLoads = kTileKeys * kKUnits / kWave;  // load instructions per tile
  constexpr int kStageBytes = kWaves * kTileKeys * kKPitch * 16;
  constexpr int kComboBytes = 2 * VEC * kWave * 16;  // the epilogue's wave-combine regions
  __shared__ __align__(16) unsigned char s_lds[kStageBytes > kComboBytes ? kStageBytes : kComboBytes];
  u32x4* s_k = reinterpret_cast<u32x4*>(s_lds) + wave * kTileKeys * kKPitch;

  const int n_tiles = (j1 - j0 + kTileKeys - 1) / kTileKeys;

  // Keys past j1 read a valid row (j0) and are masked out of the softmax.  A
  // tile index past the end re-reads the last tile (a cached read): the
  // pipeline then issues the same loads on every path, so the compiler's
  // wait counts cover exactly the tile being computed.
  auto load_tile = [&](Tile& T, int t) {
    const int jt = j0 + min(t, n_tiles - 1) * kTileKeys;
#pragma unroll
    for (int i = 0; i < kKLoads; ++i) {
      const int f = i * kWave + lane;
      const int j = jt + f / kKUnits;
      const int r = row_of(j < j1 ? j : j0);
      T.kx[i] = stream_load<u32x4>(key_row(r) + (f % kKUnits) * (16 / static_cast<int>(sizeof(KT))));
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int j = jt + 4 * grp + i;
      const int r = row_of(j < j1 ? j : j0);
      const KT* p = value_row(r) + SEG * col;
      if constexpr (F8) {
        if constexpr (VEC == 16) {
          const u32x4 x = stream_load<u32x4>(p);
#pragma unroll
          for (int w = 0; w < 4; ++w) T.vx[i][w] = x[w];
        } else if constexpr (VEC == 8) {
          const u32x2 x = stream_load<u32x2>(p);
          T.vx[i][0] = x[0];
          T.vx[i][1] = x[1];
        } else {
          T.vx[i][0] = stream_load<uint32_t>(p);
        }
      } else {
#pragma unroll
        for (int sg = 0; sg < NSEG; ++sg) {
          if constexpr (SEG == 8) {
            const u32x4 x = stream_load<u32x4>(p + sg * 16 * SEG);
#pragma unroll
            for (int w = 0; w < 4; ++w) T.vx[i][sg * 4 + w] = x[w];
          } else {
            const u32x2 x = stream_load<u32x2>(p + sg * 16 * SEG);
            T.vx[i][sg * 2] = x[0];
            T.vx[i][sg * 2 + 1] = x[1];
          }
        }
      }
    }
  };

  OnlineHeads<D, F8> st;
  st.init();
  const float sl2 = a.scale_log2;

  auto compute_tile = [&](const Tile& T, int t) {
    const int jt = j0 + t * kTileKeys;
    floatx4 s = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int i = 0; i < kKLoads; ++i) {
      const int f = i * kWave + lane;
      s_k[(f / kKUnits) * kKPitch + f % kKUnits] = T.kx[i];
    }
    if constexpr (F8) {
      // 16 codes per unit: widened to bf16 (exact), two steps each.
#pragma unroll
      for (int kk = 0; kk < D / 64; ++kk) {
        const u32x4 w = s_k[col * kKPitch + 4 * kk + grp];
        s = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, fp8x8_to_bf16x8(w[0], w[1])),
                                                    qf[2 * kk], s, 0, 0, 0);
        s = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, fp8x8_to_bf16x8(w[2], w[3])),
                                                    qf[2 * kk + 1], s, 0, 0, 0);
      }
    } else {
#pragma unroll
      for (int kk = 0; kk < KCH; ++kk)
        s = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, s_k[col * kKPitch + 4 * kk + grp]),
                                                    qf[kk], s, 0, 0, 0);
    }
    st.add(s, T.vx, jt, j1, sl2, grp);
  };

  // Two register buffers: the loads of this wave's next tile are in flight
  // while the current one is computed.  The loop body is straight-line (a
  // past-the-end prefetch re-reads the last tile), so the wait before each
  // tile covers exactly that tile's loads.
  const int my_tiles = n_tiles > wave ? (n_tiles - wave + kWaves - 1) / kWaves : 0;
  Tile T0, T1;
  load_tile(T0, wave);
  int i = 0;
  for (; i + 2 <= my_tiles; i += 2) {
    const int t = wave + i * kWaves;
    load_tile(T1, t + kWaves);
    compute_tile(T0, t);
    load_tile(T0, t + 2 * kWaves);
    compute_tile(T1, t + kWaves);
  }
  if (i < my_tiles) compute_tile(T0, wave + i * kWaves);

  // ---- combine the four waves: (m, l) per head, then O in wave order ----
  float l_run = st.l, z_run = st.z;
  const float m_run = st.m;
  l_run = sum_across_rows(l_run);
  z_run = sum_across_rows(z_run);
  __shared__ float s_m[kWaves][16];
  __shared__ float s_l[kWaves][16];
  __shared__ float s_z[kWaves][16];
  if (grp == 0) {
    s_m[wave][col] = m_run;
    s_l[wave][col] = l_run;
    s_z[wave][col] = z_run;
  }
  __syncthreads();
  float Mx = neg_inf();
#pragma unroll
  for (int w = 0; w < kWaves; ++w) Mx = fmaxf(Mx, s_m[w][col]);
  float Lx = 0.f;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) Lx += s_l[w][col] * __builtin_amdgcn_exp2f(s_m[w][col] - Mx);
  float Zx = 0.f;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) Zx += s_z[w][col] * __builtin_amdgcn_exp2f(s_m[w][col] - Mx);
  const float f = __builtin_amdgcn_exp2f(m_run - Mx);  // 0 for a wave with no tile
#pragma unroll
  for (int e = 0; e < VEC; ++e) st.acc[e] *= f;
  // O of the four waves, summed as (w0 + w1) + (w2 + w3) in registers: a
  // wave stores its accumulators (16 bytes per lane and output tile, lane-
  // contiguous) and its partner adds them; two rounds over two LDS regions.
  floatx4* s_x = reinterpret_cast<floatx4*>(s_lds);
  if (wave & 1) {
#pragma unroll
    for (int e = 0; e < VEC; ++e) s_x[((wave >> 1) * VEC + e) * kWave + lane] = st.acc[e];
  }
  __syncthreads();
  if (!(wave & 1)) {
#pragma unroll
    for (int e = 0; e < VEC; ++e) st.acc[e] += s_x[((wave >> 1) * VEC + e) * kWave + lane];
  }
  __syncthreads();
  if (wave == 2) {
#pragma unroll
    for (int e = 0; e < VEC; ++e) s_x[e * kWave + lane] = st.acc[e];
  }
  __syncthreads();
  if (wave != 0) {
    store_copy();
    return;
  }
#pragma unroll
  for (int e = 0; e < VEC; ++e) st.acc[e] += s_x[e * kWave + lane];

  // Partial row item * Hkv + g: pm/pl/pz [G], po [G, D], written by
  // wave 0 from its registers (acc[e][jj] of lane (grp, col): head col,
  // d = (e / SEG) * 16 * SEG + SEG * (4 grp + jj) + e % SEG).
  const int64_t pidx = static_cast<int64_t>(item) * a.Hkv + g;
  if (col < a.G) {
    if (grp == 0) {
      a.pm[pidx * a.G + col] = Mx;
      a.pl[pidx * a.G + col] = Lx;
      a.pz[pidx * a.G + col] = Zx;
    }
    float* po = a.po + (pidx * a.G + col) * D;
#pragma unroll
    for (int sg = 0; sg < NSEG; ++sg)
#pragma unroll
      for (int jj = 0; jj < 4; ++jj)
#pragma unroll
        for (int w = 0; w < SEG / 4; ++w) {
          const int e = sg * SEG + 4 * w;
          *reinterpret_cast<floatx4*>(po + sg * 16 * SEG + SEG * (4 * grp + jj) + 4 * w) =
              floatx4{st.acc[e][jj], st.acc[e + 1][jj], st.acc[e + 2][jj], st.acc[e + 3][jj]};
        }
  }
  store_copy();
}

// ---------------------------------------------------------------------------
// Full-context attention of several new query rows per sequence (the causal
// draft-extend, row t of sequence b seeing the first lens[b] - n + t + 1
// rows).  The rows of one sequence read almost the same keys, so a work item
// is a key chunk of a sequence rather than of a row: its workgroup streams the
// chunk once through LDS and each of its eight waves attends one query row
// over it (further rows take further passes).  The chunk size and the
// numbering of each row's partials are those of the per-row decomposition
// (wave_chunk, locate_item): a row's items are the chunks it sees, and the
// same merge kernel combines them.

constexpr int kRowWaves = 8;                      // query rows per pass, one per wave
constexpr int kRowThreads = kRowWaves * kWave;
constexpr int kRowStep = kChunkQuantum;           // keys per LDS step: four 16-key tiles
constexpr int kRowGroup = 4;                      // tiles per softmax update (even: PV in tile pairs)
static_assert(kRowGroup % 2 == 0, "the multi-row kernel's PV product takes tiles in pairs");

// Finds sequence b and chunk c of multi-row work item `item`: sequence b owns
// as many items as its last row has chunks.  Also returns b's row count n and
// the number of partials numbered before b's last row.  Returns false for the
// whole workgroup when `item` lies past the last sequence's items.
__device__ bool locate_rows_item(const SplitArgs& a, int item, int& b_out, int& c_out, int& n_out,
                                 int& before_last_out, int& chunk_out) {
  constexpr KeyMap M = KeyMap::Full;
  __shared__ int s_b, s_c, s_n, s_before, s_chunk;
  const int NV = a.B * a.qps;
  if (threadIdx.x < kWave) {
    const int lane = threadIdx.x;
    int first;
    const int chunk = wave_chunk<M>(a.lens, a.n_q, a.qps, NV, a.len_cap, a.W, a.sink, a.target,
                                    a.chunk_cap, a.err, true, a.dd, a.per_seq != 0, first);
    if (lane == 0) {
      s_b = -1;
      s_chunk = chunk;
    }
    int carry_items = 0, carry_parts = 0;
    for (int base = 0; base < NV; base += kWave) {
      const int v = base + lane;
      int cnt = 0, own = 0, b = 0, n = 0;
      if (v < NV) {
        b = a.qps == 1 ? v : v / a.qps;
        const int S =
            base == 0 ? first : visible_len<M>(a.lens, a.n_q, a.qps, a.len_cap, a.err, v, false, b, a.dd);
        cnt = ceil_div_i(S, chunk);
        n = a.n_q == nullptr ? a.qps : min(max(a.n_q[b], 0), a.qps);
        own = v - b * a.qps == n - 1 ? cnt : 0;  // the last row: the sequence's items
      }
      int incl_own = own, incl_cnt = cnt;
#pragma unroll
      for (int off = 1; off < kWave; off <<= 1) {
        const int x = __shfl_up(incl_own, off);
        const int y = __shfl_up(incl_cnt, off);
        if (lane >= off) {
          incl_own += x;
          incl_cnt += y;
        }
      }
      const int lo = carry_items + incl_own - own;
      if (own > 0 && item >= lo && item < lo + own) {
        s_b = b;
        s_c = item - lo;
        s_n = n;
        s_before = carry_parts + incl_cnt - cnt;
      }
      carry_items += __shfl(incl_own, kWave - 1);
      carry_parts += __shfl(incl_cnt, kWave - 1);
      if (carry_items > item) break;
    }
  }
  __syncthreads();
  b_out = s_b;
  c_out = s_c;
  n_out = s_n;
  before_last_out = s_before;
  chunk_out = s_chunk;
  return b_out >= 0;
}

// Instruction order of a run of N LDS operand reads, each feeding R MFMAs:
// the first kAhead reads go out before any of the run's MFMAs and every
// later read follows the MFMAs of the operand read kAhead before it, so
// kAhead reads are in flight while the MFMAs run (left to itself the
// scheduler kept one or two).  Measured on the multi-row kernel: kAhead 5
// took 8 rows at 1M from 506-520 to 487-490 us (8 and 12 gained less, 12
// lost ground at 3 rows).
template <int N, int R>
__device__ __forceinline__ void pipeline_lds_reads() {
  constexpr int kAhead = N < 5 ? N : 5;
  constexpr int kDsRead = 0x100, kMfma = 0x008;  // sched_group_barrier instruction classes
#pragma unroll
  for (int i = 0; i < kAhead; ++i) __builtin_amdgcn_sched_group_barrier(kDsRead, 1, 0);
#pragma unroll
  for (int i = kAhead; i < N; ++i) {
    __builtin_amdgcn_sched_group_barrier(kMfma, R, 0);
    __builtin_amdgcn_sched_group_barrier(kDsRead, 1, 0);
  }
  __builtin_amdgcn_sched_group_barrier(kMfma, R * kAhead, 0);
}

// F8: the cache holds E4M3 codes; a step's codes are widened to bf16 when
// they are stored into LDS (the same layouts as for a bf16 cache), so the
// compute is the same; the key scale is folded into the logit scale and the
// value scale into the merge's normalisation.
template <int D, bool F8>
__global__ __launch_bounds__(kRowThreads) void rows_split_kernel(SplitArgs a) {
  constexpr KeyMap M = KeyMap::Full;
  using KT = std::conditional_t<F8, uint8_t, uint16_t>;  // one cached K/V element
  constexpr int VEC = D / 16;
  constexpr int SEG = VEC < 8 ? VEC : 8;  // as in split_kernel
  constexpr int NSEG = VEC / SEG;
  constexpr int KCH = D / 32;
  constexpr int kUnits = D / 8;  // 16-byte bf16 units per row of one KV head (in LDS)
  // K rows are staged key-major at a pitch of kUnits + 2 units: the K
  // operand read (16 lanes take one unit of 16 rows) is then free of bank
  // conflicts on gfx950.
  constexpr int kPitch = kUnits + 2;
  constexpr int kLUnits = F8 ? D / 16 : kUnits;  // 16-byte units per row as loaded (codes or bf16)
  constexpr int kLoads = kRowStep * kLUnits / kRowThreads;  // K (and V) units per thread and step
  static_assert(kRowStep == 64, "rows_kernel_fits assumes 64-key steps");
  static_assert(kLoads == 1 || kLoads == 2 || kLoads == 4, "a thread's keys must sit in one 4-key run");
  static_assert(kRowStep * kUnits % kRowThreads == 0, "step must tile the workgroup");
  // V is staged transposed, in the order of the PV product's operand: one
  // LDS row per value column d, holding the step's 64 keys as
  // k' = 32 pair + 8 grp + 4 (tile % 2) + i for key 4 grp + i of tile
  // 2 pair + tile % 2.  A 16x16x32 MFMA then takes two tiles at once: its
  // 32-key index 8 grp + i stands for key 4 grp + i % 4 of tile i / 4, so
  // each lane's weights (P^T operand) are its own of both tiles, and the
  // output layout is that of the 16-key product.  Lane (grp, col)
  // then reads the operand of output tile e of segment sg (value column
  // d = 16 SEG sg + SEG col + e, keys 8 grp .. 8 grp + 7 of a tile pair) as
  // one 16-byte unit, with no byte permutes: the transposition is done once
  // per workgroup when the rows are stored, not once per query row.  Row
  // r(d) = (NSEG e + sg) * 16 + col puts the 16 lanes of one read on 16
  // consecutive rows; an odd pitch (8 units of keys + 1) keeps those reads
  // free of bank conflicts.
  constexpr int kVTPitch = kRowStep * 2 / 16 + 1;
  // Two buffers of one step's K and V rows: a step is computed from one while
  // the next step's rows, loaded during that computation, go to the other.
  __shared__ u32x4 s_k[2][kRowStep * kPitch];
  __shared__ u32x4 s_vt[2][D * kVTPitch];

  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int grp = lane >> 4;
  const int col = lane & 15;
  const int g = blockIdx.x % a.Hkv;
  const int item = blockIdx.x / a.Hkv;

  int b, c, n, before_last, chunk;
  if (!locate_rows_item(a, item, b, c, n, before_last, chunk)) return;
  b = __builtin_amdgcn_readfirstlane(b);
  c = __builtin_amdgcn_readfirstlane(c);
  n = __builtin_amdgcn_readfirstlane(n);
  before_last = __builtin_amdgcn_readfirstlane(before_last);
  chunk = __builtin_amdgcn_readfirstlane(chunk);
  auto row_len = [&](int t) {
    int bb;
    return visible_len<M>(a.lens, a.n_q, a.qps, a.len_cap, a.err, b * a.qps + t, false, bb, a.dd);
  };
  const int S = __builtin_amdgcn_readfirstlane(row_len(n - 1));  // the last row sees every key
  const int j0 = c * chunk;
  const int j1 = min(j0 + chunk, S);
  const int n_steps = ceil_div_i(j1 - j0, kRowStep);

  const int64_t rs = static_cast<int64_t>(a.Hkv) * D;
  const int64_t seq_off = (static_cast<int64_t>(b) * a.rows * a.Hkv + g) * D;
  const KT* kbase = static_cast<const KT*>(a.k) + seq_off;
  const KT* vbase = static_cast<const KT*>(a.v) + seq_off;

  // Thread tid holds loaded unit tid % kLUnits of the kLoads consecutive keys
  // kLoads * (tid / kLUnits) + i of a step (a run inside one 4-key group of a
  // tile); the lanes of a load instruction cover whole rows of several keys.
  // A load addresses the step's first row (wave-uniform) plus a fixed 32-bit
  // byte offset per thread and key; keys past j1 read the step's first row
  // (masked out of every row's softmax).
  const int my_unit = tid % kLUnits;
  const int my_key0 = kLoads * (tid / kLUnits);
  const uint32_t row_bytes = static_cast<uint32_t>(rs) * sizeof(KT);  // one token row, all KV heads
  uint32_t my_off[kLoads];
#pragma unroll
  for (int i = 0; i < kLoads; ++i) my_off[i] = (my_key0 + i) * row_bytes + my_unit * 16u;
  // Where this thread's keys and value columns land in the transposed V:
  // k' of its first key, and the row of value column 8 my_unit + x.
  const int my_kq = ((my_key0 >> 5) << 5) + ((my_key0 & 15) >> 2) * 8 + ((my_key0 >> 4) & 1) * 4 + (my_key0 & 3);
  auto vt_row = [](int dd) { return ((dd % SEG) * NSEG + dd / (16 * SEG)) * 16 + (dd / SEG) % 16; };
  u32x4 rk[kLoads], rv[kLoads];
  auto load = [&](int s) {
    const int js = j0 + s * kRowStep;
    const int64_t step_off = static_cast<int64_t>(js) * row_bytes;
    const char* ks = reinterpret_cast<const char*>(kbase) + step_off;
    const char* vs = reinterpret_cast<const char*>(vbase) + step_off;
    const int left = j1 - js;  // keys of the chunk from this step on (wave-uniform)
    if (left >= kRowStep) {
#pragma unroll
      for (int i = 0; i < kLoads; ++i) {
        rk[i] = stream_load<u32x4>(ks + my_off[i]);
        rv[i] = stream_load<u32x4>(vs + my_off[i]);
      }
    } else {
#pragma unroll
      for (int i = 0; i < kLoads; ++i) {
        const uint32_t off = my_key0 + i < left ? my_off[i] : my_unit * 16u;
        rk[i] = stream_load<u32x4>(ks + off);
        rv[i] = stream_load<u32x4>(vs + off);
      }
    }
  };
  auto stash = [&](int buf) {
    if constexpr (F8) {
      // 16 codes per unit: K widened into two bf16 units of its row; V
      // column by column (16 my_unit + x) into the transposed rows.
#pragma unroll
      for (int i = 0; i < kLoads; ++i) {
        u32x4* dst = s_k[buf] + (my_key0 + i) * kPitch + 2 * my_unit;
        dst[0] = fp8x8_to_bf16x8(rk[i][0], rk[i][1]);
        dst[1] = fp8x8_to_bf16x8(rk[i][2], rk[i][3]);
      }
      unsigned char* vt = reinterpret_cast<unsigned char*>(s_vt[buf]) + my_kq * 2;
      auto widen = [](uint32_t w, int x) {  // codes x & ~1, x | 1 of word w -> two bf16 (x & 2 picks the half)
        return (x & 2) ? fp8x2_to_bf16x2<true>(w) : fp8x2_to_bf16x2<false>(w);
      };
#pragma unroll
      for (int x = 0; x < 16; ++x) {
        unsigned char* dst = vt + vt_row(16 * my_unit + x) * (kVTPitch * 16);
        const uint32_t b0 = widen(rv[0][x >> 2], x);
        if constexpr (kLoads == 2) {
          const uint32_t b1 = widen(rv[1][x >> 2], x);
          *reinterpret_cast<uint32_t*>(dst) = __builtin_amdgcn_perm(b1, b0, (x & 1) ? 0x07060302u : 0x05040100u);
        } else {
          static_assert(kLoads == 1, "fp8 runs are one or two keys");
          *reinterpret_cast<uint16_t*>(dst) = static_cast<uint16_t>(b0 >> (16 * (x & 1)));
        }
      }
      return;
    }
#pragma unroll
    for (int i = 0; i < kLoads; ++i) s_k[buf][(my_key0 + i) * kPitch + my_unit] = rk[i];
    unsigned char* vt = reinterpret_cast<unsigned char*>(s_vt[buf]) + my_kq * 2;
#pragma unroll
    for (int x = 0; x < 8; ++x) {  // value column 8 my_unit + x: this thread's keys, in k' order
      const int w = x >> 1;
      unsigned char* dst = vt + vt_row(8 * my_unit + x) * (kVTPitch * 16);
      if constexpr (kLoads == 4) {
        const uint32_t sel = (x & 1) ? 0x07060302u : 0x05040100u;
        *reinterpret_cast<u32x2*>(dst) = u32x2{__builtin_amdgcn_perm(rv[1][w], rv[0][w], sel),
                                               __builtin_amdgcn_perm(rv[3][w], rv[2][w], sel)};
      } else if constexpr (kLoads == 2) {
        const uint32_t sel = (x & 1) ? 0x07060302u : 0x05040100u;
        *reinterpret_cast<uint32_t*>(dst) = __builtin_amdgcn_perm(rv[1][w], rv[0][w], sel);
      } else {
        *reinterpret_cast<uint16_t*>(dst) = static_cast<uint16_t>(rv[0][w] >> (16 * (x & 1)));
      }
    }
  };
  // weigh_lean takes a positive scale: a negative one is applied as its
  // magnitude with the queries negated (exact in bf16), zero as the smallest
  // normal float.
  const float sl2 = fmaxf(fabsf(a.scale_log2), __FLT_MIN__);
  const uint32_t q_sign = a.scale_log2 < 0.f ? 0x80008000u : 0u;

  for (int t0 = 0; t0 < n; t0 += kRowWaves) {
    const int t = t0 + wave;
    const int L = t < n ? row_len(t) : 0;
    const bool active = L > j0;  // the row sees keys of this chunk
    if (!__syncthreads_or(active)) continue;
    const int j_end = min(j1, L);

    // Q^T operand of row t, laid out as in split_kernel.
    bf16x8 qf[KCH];
    {
      const bool live = active && col < a.G;
      const uint16_t* qp =
          a.q + ((static_cast<int64_t>(b) * a.qps + (active ? t : 0)) * a.Hq + g * a.G + (col < a.G ? col : 0)) * D;
#pragma unroll
      for (int kk = 0; kk < KCH; ++kk) {
        u32x4 w = live ? *reinterpret_cast<const u32x4*>(qp + kk * 32 + grp * 8) : u32x4{0u, 0u, 0u, 0u};
        qf[kk] = __builtin_bit_cast(bf16x8, w ^ q_sign);
      }
    }

    OnlineHeads<D, false> st;
    st.init();
    // A thread issues the next step's loads as soon as it has stored the
    // current ones (before the barrier), so they have the wait at the
    // barrier as well as a step of compute to arrive in.
    load(0);
    stash(0);
    if (n_steps > 1) load(1);
    __syncthreads();
    for (int s = 0; s < n_steps; ++s) {
      const int buf = s & 1;
      if (active) {
        const u32x4* sk = s_k[buf];
        const u32x4* svt = s_vt[buf];
        constexpr int NT = kRowGroup;
#pragma unroll
        for (int u0 = 0; u0 < kRowStep / kTileKeys; u0 += NT) {
          const int js = j0 + s * kRowStep + u0 * kTileKeys;
          if (js >= j_end) break;  // past this row's last key (wave-uniform)
          // Logits of NT tiles: independent MFMA chains.
          floatx4 sc[NT];
#pragma unroll
          for (int u = 0; u < NT; ++u) sc[u] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int kk = 0; kk < KCH; ++kk)
#pragma unroll
            for (int u = 0; u < NT; ++u)
              sc[u] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                  __builtin_bit_cast(bf16x8, sk[((u0 + u) * kTileKeys + col) * kPitch + 4 * kk + grp]), qf[kk],
                  sc[u], 0, 0, 0);
          pipeline_lds_reads<KCH * NT, 1>();
          bf16x4 pop[NT];
          st.template weigh_lean<NT>(sc, js, j_end, sl2, grp, pop);
          // O^T += V^T . P^T over tile pairs: output tile sg * SEG + e takes
          // the transposed V unit of value column 16 SEG sg + SEG col + e,
          // keys 8 grp .. 8 grp + 7 of the pair.
#pragma unroll
          for (int u = 0; u < NT; u += 2) {
            const bf16x8 pp = __builtin_shufflevector(pop[u], pop[u + 1], 0, 1, 2, 3, 4, 5, 6, 7);
            const int unit = 2 * (u0 + u) + grp;  // 16-byte unit of keys 8 grp.. of pair (u0 + u) / 2
#pragma unroll
            for (int sg = 0; sg < NSEG; ++sg)
#pragma unroll
              for (int e = 0; e < SEG; ++e) {
                const u32x4 w = svt[((e * NSEG + sg) * 16 + col) * kVTPitch + unit];
                st.acc[sg * SEG + e] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, w), pp,
                                                                                st.acc[sg * SEG + e], 0, 0, 0);
              }
            pipeline_lds_reads<NSEG * SEG, 1>();
          }
        }
      }
      if (s + 1 < n_steps) {
        stash(buf ^ 1);
        if (s + 2 < n_steps) load(s + 2);
      }
      __syncthreads();
    }

    if (active) {
      // This row's partial: its items are numbered after those of every
      // earlier row; rows t .. n-2 precede the last one.
      int later = 0;
      for (int t2 = t + lane; t2 < n - 1; t2 += kWave) later += ceil_div_i(row_len(t2), chunk);
#pragma unroll
      for (int off = kWave / 2; off > 0; off >>= 1) later += __shfl_xor(later, off);
      float l = st.l, z = st.z;
      l = sum_across_rows(l);
      z = sum_across_rows(z);
      const int64_t pidx = static_cast<int64_t>(before_last - later + c) * a.Hkv + g;
      if (col < a.G) {
        if (grp == 0) {
          a.pm[pidx * a.G + col] = st.m;
          a.pl[pidx * a.G + col] = l;
          a.pz[pidx * a.G + col] = z;
        }
        float* po = a.po + (pidx * a.G + col) * D;
#pragma unroll
        for (int sg = 0; sg < NSEG; ++sg)
#pragma unroll
          for (int jj = 0; jj < 4; ++jj)
#pragma unroll
            for (int w = 0; w < SEG / 4; ++w) {
              const int e = sg * SEG + 4 * w;
              *reinterpret_cast<floatx4*>(po + sg * 16 * SEG + SEG * (4 * grp + jj) + 4 * w) =
                  floatx4{st.acc[e][jj], st.acc[e + 1][jj], st.acc[e + 2][jj], st.acc[e + 3][jj]};
            }
      }
    }
  }
}

// One workgroup of NT threads per (b, h, SLICE-wide slice of d).  Thread t
// owns float4 column q4 = t % (SLICE/4) of the slice and item slot
// t / (SLICE/4); the slots walk the sequence's items (several loads in flight
// per thread), then are summed by a fixed-order tree in LDS, so the result
// does not depend on timing.  Two shapes: 1024 threads on 64-wide slices for
// sequences with many items (one long sequence), 256 threads on whole rows
// when items per sequence are few (many short windows).
template <int D, KeyMap M, int NT, int SLICE>
__global__ __launch_bounds__(NT) void merge_kernel(MergeArgs a) {
  constexpr int Q = SLICE / 4;  // float4 columns per slice
  constexpr int NS = NT / Q;    // item slots
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = tid / kWave;
  const int q4 = tid % Q;
  const int slot = tid / Q;
  const int v = blockIdx.x / a.Hq;  // query row
  const int h = blockIdx.x % a.Hq;
  const int g = h / a.G;
  const int hl = h % a.G;
  const int d0 = blockIdx.y * SLICE + 4 * q4;

  __shared__ int s_base, s_cnt;
  __shared__ float s_red[NT / kWave];
  __shared__ float s_m[NS];
  __shared__ floatx4 s_o[NS][Q];
  __shared__ float s_L[NS];
  __shared__ float s_Z[NS];
  if (tid < kWave) {
    int first;
    const int chunk = wave_chunk<M>(a.lens, a.n_q, a.qps, a.B * a.qps, a.len_cap, a.W, a.sink,
                                    a.target, a.chunk_cap, a.err, false, a.dd, a.per_seq != 0, first);
    int before = 0, mine = 0;
    for (int base = 0; base <= v; base += kWave) {
      const int vv = base + lane;
      if (vv <= v) {
        int bb;
        const int S =
            base == 0 ? first : visible_len<M>(a.lens, a.n_q, a.qps, a.len_cap, a.err, vv, false, bb, a.dd);
        const int cnt = ceil_div_i(selected_count<M>(S, a.W, a.sink), chunk);
        if (vv < v) before += cnt; else mine = cnt;
      }
    }
#pragma unroll
    for (int off = kWave / 2; off > 0; off >>= 1) {
      before += __shfl_xor(before, off);
      mine += __shfl_xor(mine, off);
    }
    if (lane == 0) {
      s_base = before;
      s_cnt = mine;
    }
  }
  __syncthreads();
  const int base = s_base;
  const int n = s_cnt;
  auto prow = [&](int c) { return (static_cast<int64_t>(base + c) * a.Hkv + g) * a.G + hl; };
  if constexpr (is_step(M)) {
    // The fused step's new length; this launch reads only the old lengths.
    if (h == 0 && blockIdx.y == 0 && tid == 0) {
      int bb;
      a.lens_out[v] = visible_len<M>(a.lens, a.n_q, a.qps, a.len_cap, a.err, v, false, bb, a.dd);
    }
  }

  float Mx;  // the largest partial maximum (slot 0)
  if (n <= NS) {
    // At most one item per slot: one round of loads; the slots are combined
    // pairwise in a fixed tree order, rescaled to the larger maximum (every
    // partial has at least one key, so an item's maximum is finite).
    float m = neg_inf();
    floatx4 o = {0.f, 0.f, 0.f, 0.f};
    float L = 0.f, Z = 0.f;
    if (slot < n) {
      const int64_t pr = prow(slot);
      m = a.pm[pr];
      o = *reinterpret_cast<const floatx4*>(a.po + pr * D + d0);
      L = a.pl[pr];
      Z = a.pz[pr];
    }
    s_o[slot][q4] = o;
    if (q4 == 0) {
      s_m[slot] = m;
      s_L[slot] = L;
      s_Z[slot] = Z;
    }
    __syncthreads();
    // Round `half`: slot s < half takes in slot s + half.  Every thread of a
    // slot carries the slot's maximum in a register, so a round writes the
    // maxima of slots below `half` only and reads those at or above it.
#pragma unroll
    for (int half = NS / 2; half > 0; half >>= 1) {
      if (slot < half) {
        const float m2 = s_m[slot + half];
        if (m2 != neg_inf()) {
          const float mn = fmaxf(m, m2);
          const float f1 = __builtin_amdgcn_exp2f(m - mn);
          const float f2 = __builtin_amdgcn_exp2f(m2 - mn);
          s_o[slot][q4] = s_o[slot][q4] * f1 + s_o[slot + half][q4] * f2;
          if (q4 == 0) {
            s_m[slot] = mn;
            s_L[slot] = s_L[slot] * f1 + s_L[slot + half] * f2;
            s_Z[slot] = s_Z[slot] * f1 + s_Z[slot + half] * f2;
          }
          m = mn;
        }
      }
      __syncthreads();
    }
    Mx = m;
  } else {
    // The partials of a slot's first kPre items are loaded before the
    // largest maximum is known (they do not depend on it), so the two
    // rounds of loads overlap; items past those (rows with more than
    // kPre * NS items) are loaded in the loop below.  The loads are
    // unconditional (a slot past the row's last item re-reads that item and
    // ignores it): a load under a branch made the compiler wait for it there.
    constexpr int kPre = NS >= 32 ? 2 : 8;
    float pmv[kPre], plv[kPre], pzv[kPre];
    floatx4 pov[kPre];
    // (The maxima first: the wait for them then leaves the rest in flight.)
#pragma unroll
    for (int i = 0; i < kPre; ++i) pmv[i] = a.pm[prow(min(slot + i * NS, n - 1))];
#pragma unroll
    for (int i = 0; i < kPre; ++i) {
      const int64_t pr = prow(min(slot + i * NS, n - 1));
      pov[i] = *reinterpret_cast<const floatx4*>(a.po + pr * D + d0);
      plv[i] = a.pl[pr];
      pzv[i] = a.pz[pr];
    }
    // Largest partial maximum.
    float mx = neg_inf();
#pragma unroll
    for (int i = 0; i < kPre; ++i) mx = fmaxf(mx, slot + i * NS < n ? pmv[i] : neg_inf());
    for (int c = kPre * NS + tid; c < n; c += NT) mx = fmaxf(mx, a.pm[prow(c)]);  // the other items
#pragma unroll
    for (int off = kWave / 2; off > 0; off >>= 1) mx = fmaxf(mx, __shfl_xor(mx, off));
    if (lane == 0) s_red[wave] = mx;
    __syncthreads();
    Mx = s_red[0];
#pragma unroll
    for (int w = 1; w < NT / kWave; ++w) Mx = fmaxf(Mx, s_red[w]);

    // Items in order c = slot, slot + NS, ...
    floatx4 o = {0.f, 0.f, 0.f, 0.f};
    float L = 0.f, Z = 0.f;
#pragma unroll
    for (int i = 0; i < kPre; ++i) {
      if (slot + i * NS < n) {
        const float w = __builtin_amdgcn_exp2f(pmv[i] - Mx);
        o += w * pov[i];
        L += w * plv[i];
        Z += w * pzv[i];
      }
    }
#pragma unroll 8
    for (int c = slot + kPre * NS; c < n; c += NS) {
      const int64_t pr = prow(c);
      const float w = __builtin_amdgcn_exp2f(a.pm[pr] - Mx);
      const floatx4 v = *reinterpret_cast<const floatx4*>(a.po + pr * D + d0);
      o += w * v;
      L += w * a.pl[pr];
      Z += w * a.pz[pr];
    }
    s_o[slot][q4] = o;
    if (q4 == 0) {
      s_L[slot] = L;
      s_Z[slot] = Z;
    }
    __syncthreads();
#pragma unroll
    for (int half = NS / 2; half > 0; half >>= 1) {
      if (slot < half) {
        s_o[slot][q4] += s_o[slot + half][q4];
        if (q4 == 0) {
          s_L[slot] += s_L[slot + half];
          s_Z[slot] += s_Z[slot + half];
        }
      }
      __syncthreads();
    }
  }
  if (slot == 0) {
    const float Lt = s_L[0];
    const floatx4 ot = s_o[0][q4];
    float r[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) r[i] = n > 0 ? ot[i] / Lt * a.out_scale : 0.f;
    const uint32_t lo = pack_bf16x2(r[0], r[1]);
    const uint32_t hi = pack_bf16x2(r[2], r[3]);
    *reinterpret_cast<u32x2*>(a.out + (static_cast<int64_t>(v) * a.Hq + h) * D + d0) = u32x2{lo, hi};
    if (a.lse != nullptr && blockIdx.y == 0 && q4 == 0)
      a.lse[static_cast<int64_t>(v) * a.Hq + h] = n > 0 ? (Mx + log2f(s_Z[0])) * kLn2 : neg_inf();
  }
}

template <int D, KeyMap M, bool F8>
hipError_t launch_typed(const AttnLaunch& L, hipStream_t st) {
  const int G = L.Hq / L.Hkv;
  if (L.max_items > 0) {
    SplitArgs a;
    a.q = L.q; a.k = L.k; a.v = L.v; a.lens = L.lens; a.n_q = L.n_q; a.qps = L.qps;
    a.table = L.table; a.table_stride = L.table_stride;
    a.pm = L.pm; a.pl = L.pl; a.pz = L.pz; a.po = L.po; a.err = L.err;
    a.B = L.B; a.Hq = L.Hq; a.Hkv = L.Hkv; a.G = G;
    a.rows = L.rows; a.len_cap = L.len_cap;
    a.W = L.W; a.sink = L.sink; a.R_w = L.R_w;
    a.target = L.target; a.chunk_cap = L.chunk_cap;
    a.scale_log2 = L.scale * L.k_scale * kLog2e;
    a.k2 = L.k2; a.v2 = L.v2; a.rows2 = L.rows2; a.dd = L.dd;
    a.per_seq = L.per_seq ? 1 : 0;
    if constexpr (M == KeyMap::Full && (!F8 || D >= 128)) {
      if (L.qps > 1 && rows_kernel_fits(L.Hkv, L.d, F8)) {
        // Items of the multi-row kernel: sequence b owns ceil(n(b) / chunk)
        // of them, n(b) its last row's length; with the chunk of the per-row
        // decomposition (total over rows / T, clamped to [quantum, cap]) that
        // is at most min(B ceil(n/quantum), max(T + B, B ceil(n/cap))).
        const int64_t n = L.len_cap;
        const int64_t fine = static_cast<int64_t>(L.B) * ((n + kChunkQuantum - 1) / kChunkQuantum);
        const int64_t coarse = static_cast<int64_t>(L.B) * ((n + L.chunk_cap - 1) / L.chunk_cap);
        const int64_t items = std::min(fine, std::max<int64_t>(static_cast<int64_t>(L.target) + L.B, coarse));
        const dim3 grid(static_cast<unsigned>(std::min<int64_t>(items, L.max_items)) * static_cast<unsigned>(L.Hkv));
        hipLaunchKernelGGL((rows_split_kernel<D, F8>), grid, dim3(kRowThreads), 0, st, a);
      } else {
        hipLaunchKernelGGL((split_kernel<D, M, F8>), dim3(static_cast<unsigned>(L.max_items) * L.Hkv),
                           dim3(kThreads), 0, st, a);
      }
    } else {
      const dim3 grid(static_cast<unsigned>(L.max_items) * static_cast<unsigned>(L.Hkv));
      hipLaunchKernelGGL((split_kernel<D, M, F8>), grid, dim3(kThreads), 0, st, a);
    }
  }
  // The merge shape: 1024-thread workgroups on 64-wide slices when a row has
  // many items and their grid fits one workgroup per CU; for full-context
  // rows (O(S) items each) whose wide grid does not fit, 512-thread
  // workgroups on 128-wide slices (sixteen item slots: a row's first 128
  // items in one round of loads) while two of them per CU hold the grid (a
  // tree of 4 candidates took 4.6 -> 5.1 us on it); else one 256-thread workgroup
  // per row and head (a tree of 4 speculation candidates at Hq = 32, 512
  // wide workgroups: 22.4 -> 20.8 us per draft step).
  const int64_t NV = static_cast<int64_t>(L.B) * L.qps;
  const bool many = L.max_items >= 32 * NV;
  const bool wide = many && NV * L.Hq * (D / 64) <= static_cast<int64_t>(device_cus());
  const bool mid = many && !wide && !is_windowed(M) && D >= 128 &&
                   NV * L.Hq * (D / 128) <= 2 * static_cast<int64_t>(device_cus());
  MergeArgs m;
  m.lens = L.lens; m.n_q = L.n_q; m.qps = L.qps; m.pm = L.pm; m.pl = L.pl; m.pz = L.pz; m.po = L.po;
  m.out = L.out; m.lse = L.lse; m.err = L.err;
  m.B = L.B; m.Hq = L.Hq; m.Hkv = L.Hkv; m.G = G;
  m.len_cap = L.len_cap; m.W = L.W; m.sink = L.sink;
  m.target = L.target; m.chunk_cap = L.chunk_cap;
  m.out_scale = L.v_scale;
  m.dd = L.dd;
  m.lens_out = L.lens_out;
  m.per_seq = L.per_seq ? 1 : 0;
  const unsigned bh = static_cast<unsigned>(NV) * static_cast<unsigned>(L.Hq);
  if (wide) {
    hipLaunchKernelGGL((merge_kernel<D, M, kMergeThreads, 64>), dim3(bh, D / 64), dim3(kMergeThreads), 0,
                       st, m);
  } else if (mid) {
    if constexpr (D >= 128)
      hipLaunchKernelGGL((merge_kernel<D, M, 512, 128>), dim3(bh, D / 128), dim3(512), 0, st, m);
  } else {
    hipLaunchKernelGGL((merge_kernel<D, M, 256, D>), dim3(bh, 1), dim3(256), 0, st, m);
  }
  return hipGetLastError();
}

template <int D>
hipError_t launch_d(const AttnLaunch& L, hipStream_t st) {
  if (L.kv_fp8) {
    switch (L.variant) {
      case WMTP_VARIANT_FULL: return launch_typed<D, KeyMap::Full, true>(L, st);
      case WMTP_VARIANT_WINDOWED: return launch_typed<D, KeyMap::Window, true>(L, st);
      case WMTP_VARIANT_RING: return launch_typed<D, KeyMap::Ring, true>(L, st);
      case WMTP_VARIANT_PAGED_FULL: return launch_typed<D, KeyMap::PagedFull, true>(L, st);
      case WMTP_VARIANT_PAGED_WINDOWED: return launch_typed<D, KeyMap::PagedWindow, true>(L, st);
      default: return hipErrorInvalidValue;  // no fp8 tree kernels
    }
  }
  if (L.step) {
    switch (L.variant) {
      case WMTP_VARIANT_WINDOWED: return launch_typed<D, KeyMap::WindowStep, false>(L, st);
      case WMTP_VARIANT_RING: return launch_typed<D, KeyMap::RingStep, false>(L, st);
      default: return hipErrorInvalidValue;
    }
  }
  switch (L.variant) {
    case WMTP_VARIANT_FULL: return launch_typed<D, KeyMap::Full, false>(L, st);
    case WMTP_VARIANT_WINDOWED: return launch_typed<D, KeyMap::Window, false>(L, st);
    case WMTP_VARIANT_RING: return launch_typed<D, KeyMap::Ring, false>(L, st);
    case WMTP_VARIANT_PAGED_FULL: return launch_typed<D, KeyMap::PagedFull, false>(L, st);
    case WMTP_VARIANT_PAGED_WINDOWED: return launch_typed<D, KeyMap::PagedWindow, false>(L, st);
    default: return launch_typed<D, KeyMap::Tree, false>(L, st);
  }
}

int env_int(const char* name, int dflt) {
  const char* s = std::getenv(name);
  if (s == nullptr || *s == '\0') return dflt;
  const int v = std::atoi(s);
  return v > 0 ? v : dflt;
}

}  // namespace

constexpr int kMaxDevices = 64;

// Compute units of the current device, queried once per device (MI355X:
// 256 when no device is visible).
int device_cus() {
  static std::atomic<int> cache[kMaxDevices];
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) {
    (void)hipGetLastError();
    return 256;
  }
  int v = cache[dev].load(std::memory_order_relaxed);
  if (v > 0) return v;
  if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || v <= 0) {
    (void)hipGetLastError();
    v = 256;
  }
  cache[dev].store(v, std::memory_order_relaxed);
  return v;
}

SplitPlan plan_split(int variant, int B, int Hq, int Hkv, int d, int64_t n_keys_max, int qps) {
  // Aim for one split workgroup per CU (256 on MI355X), with items of at
  // most `chunk_max` keys, so that a long single sequence runs in one
  // balanced round and many or variable-length sequences are cut finely
  // enough to pack without a long tail.  Measured on MI355X against two per
  // CU (the kernel's occupancy): the 1M call 1.4% faster (fp8 cache: 3%),
  // the 128K call 3%, an 8-row windowed extend 16%, a batch of 8 rings 13%;
  // fewer items also mean fewer partials for the merge.  The kernels pick the
  // item size from the actual lengths; the workspace covers every choice they can
  // make: with per-head target T and chunk in [quantum, cap], the item count
  // is at most min(B*ceil(n/quantum), max(T + B, B*ceil(n/cap))) for B query
  // rows.  Items sized per sequence (qps > 1 rows per sequence: the
  // full-context extend) are up to qps times finer: max(qps*T + B, ...).
  static const int target_env = env_int("WMTP_TARGET_ITEMS", 0);
  static const int chunk_max = std::max(
      kChunkQuantum, env_int("WMTP_CHUNK_MAX", WMTP_CHUNK_MAX_DEFAULT) / kChunkQuantum * kChunkQuantum);
  SplitPlan p{};
  // A paged item's pool rows are staged in LDS: its size is capped.
  const int cap = (variant == WMTP_VARIANT_PAGED_FULL || variant == WMTP_VARIANT_PAGED_WINDOWED)
                      ? std::min(chunk_max, kPagedChunkMax)
                      : chunk_max;
  const int64_t wgs = target_env > 0 ? target_env : device_cus();
  const int64_t T = std::max<int64_t>(1, wgs / std::max(Hkv, 1));
  p.target = static_cast<int>(std::min<int64_t>(T, INT32_MAX / 2));
  p.chunk_cap = cap;
  int64_t items = 0;
  if (n_keys_max > 0) {
    const int64_t fine = static_cast<int64_t>(B) * ((n_keys_max + kChunkQuantum - 1) / kChunkQuantum);
    const int64_t coarse = static_cast<int64_t>(B) * ((n_keys_max + cap - 1) / cap);
    items = std::min(fine, std::max(static_cast<int64_t>(std::max(qps, 1)) * T + B, coarse));
  }
  p.max_items = static_cast<int>(std::min<int64_t>(items, INT32_MAX));
  const size_t rows = static_cast<size_t>(p.max_items) * Hkv * (Hq / Hkv);
  auto up = [](size_t x) { return (x + 255) / 256 * 256; };
  p.off_pm = kTicketBytes;
  p.off_pl = p.off_pm + up(rows * sizeof(float));
  p.off_pz = p.off_pl + up(rows * sizeof(float));
  p.off_po = p.off_pz + up(rows * sizeof(float));
  p.bytes = rows ? p.off_po + up(rows * static_cast<size_t>(d) * sizeof(float)) : 0;
  return p;
}

hipError_t launch_attention(const AttnLaunch& L, hipStream_t st) {
  // Windowed calls with few query rows run the one-launch windowed kernel.
  if (L.win_items > 0) return launch_window(L, st);
  switch (L.d) {
    case 64: return launch_d<64>(L, st);
    case 128: return launch_d<128>(L, st);
    default: return launch_d<256>(L, st);
  }
}

}  // namespace wmtp
